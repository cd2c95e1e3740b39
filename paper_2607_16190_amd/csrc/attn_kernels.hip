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
// Scheduling: a persistent grid (2 workgroups per CU) pulls items from one
// queue per XCD. plan_kernel cuts every head's query blocks into 8 runs of
// equal kept-block cost, run x into queue x, heads in decreasing cost, so the
// XCDs stay balanced by construction, work on the same head together (its K/V
// stay in the shared last-level cache) and the workgroups resident on one XCD
// work on neighbouring query blocks (their kept K/V overlap in L2). A
// workgroup whose queue is empty steals from the others. FVA_SCHED_NAIVE
// launches the same item body once per item in head-major order.
//
// Query-block pairs: blocks of at most 64 real tokens (partial boxes at the
// end of an axis, or every block of a 64-token tiling) fill only two of the
// four waves, and a CU's other workgroup cannot use the idle SIMDs because
// its own waves move in step through their barriers. Two such neighbours
// (x-neighbours, else y-neighbours) run as one item instead: each on two
// waves, over the union of their kept lists (neighbouring blocks keep nearly
// the same key blocks), so every SIMD works and each K/V tile is staged once
// for both.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <type_traits>

#include "fva_common.h"
#include "fva_geometry.h"
#include "fva_internal.h"

namespace fva {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int kAttnThreads = 256;
constexpr int kRowBytes = 256;                 // one 128-dim bf16 row
constexpr int kTileBytes = 128 * kRowBytes;    // 32 KB per K or V tile
// Partial result of one chunk of a split row: O^T accumulators as
// [128 query rows][128 dims] fp32, then the exponent reference and the sum of
// P of every query row (fp32 [128] each).
constexpr int kPartialFloats = 128 * 128 + 2 * 128;

struct BlockMap;

struct AttnParams {
  const uint16_t* Q;
  const uint16_t* K;
  const uint16_t* V;
  const unsigned char* V8;  // E4M3 V tiles (FP8 variant)
  const int32_t* vexp;      // their per-channel exponents
  uint16_t* O;
  int heads;
  int64_t sb, sh, sn;
  Geometry g;
  const int32_t* counts;
  const int32_t* kv_idx;
  const BlockMap* bmap;  // [nb] block records
  const int4* chunks;    // [chunks] (row, first kept entry, end, 0) of split rows
  float* partials;       // [chunks][kPartialFloats] unnormalised O, reference, sum
  // Query-block pairs (null: none). plist holds, per pair slot, the union of
  // the two rows' kept lists in ascending block order, each entry
  // j | (not kept by the first block) << 16 | (not kept by the second) << 17;
  // pcount its length; psplit the chunk size of the plan (a pair is formed
  // only when neither row is split).
  const int32_t* plist;
  const int32_t* pcount;
  const int32_t* psplit;
  int pairs_head;        // pair slots per head
  int64_t n_rows;        // batch * heads * nb
  int trace_chunks;      // chunk records the trace holds after the rows
  float c2;  // softmax scale * log2(e)
  int64_t* trace;
};

// LDS row order of a K / V tile. Key kap = 32kg + 8g + 4hh + r is stored in
// row 32kg + 16hh + 4g + r, so that the S^T accumulator rows held by lane
// group g in tiles 2kg and 2kg+1 are the 8 consecutive keys 32kg + 8g + 0..7
// (the B operand of the PV product), and the 16 rows read by one transposing
// V load are consecutive.
__device__ __forceinline__ int key_of_row(int rho) {
  return ((rho >> 5) << 5) | (((rho >> 2) & 3) << 3) | (((rho >> 4) & 1) << 2) | (rho & 3);
}

// Uniform per-block constants for mapping a packed row index to its token,
// one 32-byte record per block in the attention workspace (block_table_kernel
// fills it once per launch, so the block loop does no integer division).
struct BlockMap {
  int tbase;      // token of the box origin
  int plane, ex;  // ey*ex and ex
  int mp, mx;     // ceil(2^16 / plane), ceil(2^16 / ex): exact quotients for rows < 128
  int n;          // real tokens
  int pslot;      // query-block pair this block starts (slot within a head), or -1
  int poff;       // block-id offset of its pair partner (> 0: it starts the pair), 0: none
};
static_assert(sizeof(BlockMap) == 32, "one scalar load per record");

__device__ __forceinline__ BlockMap block_map(const Geometry& g, int j) {
  const BlockBox b = block_box(g, j);
  BlockMap m;
  m.tbase = (b.t0 * g.H + b.y0) * g.W + b.x0;
  m.plane = b.ey * b.ex;
  m.ex = b.ex;
  m.mp = (65536 + m.plane - 1) / m.plane;
  m.mx = (65536 + m.ex - 1) / m.ex;
  m.n = b.n;
  m.pslot = -1;  // numbered by block_table_kernel
  m.poff = pair_partner(g, j);
  return m;
}

// Record of block j through the scalar cache (the kernels never write it).
__device__ __forceinline__ BlockMap load_block_map(const BlockMap* table, int j) {
  typedef __attribute__((address_space(4))) const int32_t const_i32;
  const const_i32* t = (const const_i32*)(table + j);
  BlockMap m;
  m.tbase = t[0];
  m.plane = t[1];
  m.ex = t[2];
  m.mp = t[3];
  m.mx = t[4];
  m.n = t[5];
  m.pslot = -1;  // (the block loop reads no pair fields)
  m.poff = 0;
  return m;
}

// Token of packed row r (< 128) of a block: 24-bit multiplies only.
__device__ __forceinline__ int row_token(const BlockMap& m, int r, int HW, int W) {
  const int lt = (int)(__umul24(r, m.mp) >> 16);
  const int rem = r - (int)__umul24(lt, m.plane);
  const int ly = (int)(__umul24(rem, m.mx) >> 16);
  const int lx = rem - (int)__umul24(ly, m.ex);
  return m.tbase + (int)__umul24(lt, HW) + (int)__umul24(ly, W) + lx;
}

__device__ __forceinline__ uint32_t hw_location() {
  uint32_t hw, xcc;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
  return ((xcc & 0xffu) << 16) | (hw & 0xffffu);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

typedef __attribute__((address_space(3))) void lds_void;

// Byte offsets (relative to the head base) of the 8 LDS rows this lane
// fills: wave w fills rows 32w .. 32w+31 (key group w), four rows per load
// instruction, so the lane's u-th row holds key
// kap = 32w + 8(u%4) + 4(u/4) + lane/16. Padding rows repeat the last real
// row (finite values; their scores are masked).
__device__ __forceinline__ void row_offsets(const AttnParams& P, const BlockMap& m, int (&roff)[8]) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int lq = lane >> 4;
  const int sn2 = 2 * (int)P.sn;  // bytes per token row
  const int W = P.g.W;
  const int HW = P.g.H * P.g.W;
  if (m.n == 128 && m.plane == 64 && m.ex == 8) {
    // Two full 8x8 planes: kap / 64 = w / 2, (kap / 8) % 8 = 4(w % 2) + u % 4,
    // kap % 8 = 4(u / 4) + lq, and every row is real. Other blocks (a single
    // plane included) take the general path, whose rows past n repeat the
    // last real row.
    const int a = (m.tbase + (w >> 1) * HW + 4 * (w & 1) * W) * sn2;  // wave-uniform
    const int l = lq * sn2;
#pragma unroll
    for (int u = 0; u < 8; ++u) roff[u] = a + ((u & 3) * W + 4 * (u >> 2)) * sn2 + l;
  } else if (m.n == m.ex) {
    // One line of consecutive tokens (a one-dimensional block, such as a run
    // of the Hilbert curve): key kap is token tbase + kap, clamped to the
    // last real row.
    const int last = m.n - 1;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int kap = min(32 * w + 8 * (u & 3) + 4 * (u >> 2) + lq, last);
      roff[u] = (m.tbase + kap) * sn2;
    }
  } else {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int rho = w * 32 + u * 4 + lq;
      const int kap = min(key_of_row(rho), m.n - 1);
      roff[u] = row_token(m, kap, HW, W) * sn2;
    }
  }
}

// Asynchronous global -> LDS copy of this wave's 8 KB of a tile. K rows use a
// 16-byte-chunk XOR swizzle (chunk ^ row%16), V rows an 8-byte-chunk swizzle
// (chunk8 ^ 4*(row%8)); both make the MFMA-side reads bank-conflict free.
// The copies are issued from inline assembly so that the compiler does not
// drain them (vmcnt(0)) before unrelated LDS reads; the kernel waits for them
// explicitly (wait_vmem) before the barrier that publishes a tile. M0 holds
// the LDS destination; nothing else in these kernels uses M0.
template <bool IS_V>
__device__ __forceinline__ void issue_tile(const uint16_t* __restrict__ src, const int (&roff)[8],
                                           unsigned char* tile) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int p = lane & 15;
  const int lq = lane >> 4;
  const unsigned char* gbase = reinterpret_cast<const unsigned char*>(src);  // wave-uniform
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)tile;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    // rho = 32w + 4u + lq, so rho % 16 = 4(u % 4) + lq and rho % 8 = 4(u % 2) + lq
    const int chunk = IS_V ? (p ^ (2 * (4 * (u & 1) + lq))) : (p ^ (4 * (u & 3) + lq));
    const uint32_t off = (uint32_t)roff[u] + 16u * (uint32_t)chunk;
    const uint32_t dst = lds0 + (uint32_t)((w * 8 + u) * 1024);
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(dst), "v"(off), "s"(gbase)
                 : "memory");
  }
}

// FP8 variant: asynchronous copy of this wave's 4 KB of block j's E4M3 V^T
// tile (rows = channels, 128 bytes of key positions each). Instruction u of
// wave w fills rows 8(4w + u) .. +7; lane L takes row L / 8 of them and the
// 16-byte chunk at physical position L % 8, which holds logical chunk
// (L % 8) ^ (row % 8): the reads of 16 consecutive channels at one key chunk
// then spread over all banks.
__device__ __forceinline__ void issue_v8_tile(const unsigned char* __restrict__ head, int j, unsigned char* tile) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int rr = lane >> 3;
  const uint32_t lane_off = (uint32_t)(rr * 128 + 16 * ((lane & 7) ^ rr));
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)tile;
  const uint32_t tile_off = (uint32_t)j * (uint32_t)kV8TileBytes;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int slab = 4 * w + u;
    const uint32_t off = tile_off + (uint32_t)(slab * 1024) + lane_off;
    const uint32_t dst = lds0 + (uint32_t)(slab * 1024);
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(dst), "v"(off), "s"(head)
                 : "memory");
  }
}

__device__ __forceinline__ bf16x8 to_bf16x8(f32x4 a, f32x4 b) {
  const f32x8 v = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_convertvector(v, bf16x8);
}

// Calls f(integral_constant<int, u>) for u = B .. E - 1 (compile-time steps).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Key groups (of 32) a block is processed with: the first 64-key half is
// always whole, the second holds the remaining groups (none, one or two);
// keys past n are masked. Each half runs with constant loop bounds.
__device__ __forceinline__ int ngroups_of(int n) { return n <= 64 ? 2 : (n <= 96 ? 3 : 4); }

// max over lanes l, l^16, l^32, l^48 (the four lane groups holding one
// query row) with the gfx950 lane-swap instructions; no LDS traffic.
__device__ __forceinline__ float row_max4(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Workgroup barrier without a memory fence: the only cross-wave traffic in
// the block loop is the LDS tiles written by global->LDS copies, and every
// wave waits for its own copies (vmcnt) before arriving here.
__device__ __forceinline__ void tile_barrier() { asm volatile("s_barrier" ::: "memory"); }

typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// S^T tiles of one 64-key half: LDS tiles 4hb .. 4hb + 2*NGH - 1 against the
// two 16-row Q tiles. The fragments of tile t+1 load while tile t multiplies
// (two fragment buffers, renamed at compile time).
// One work item: query block `row` (= (b * heads + h) * nb + i) against the
// kept-list entries [begin, end) of its row. partial == nullptr: the whole
// row, normalised into O; otherwise one chunk of a split row, whose
// unnormalised result goes to partial for the combine step. pslot >= 0: the
// query-block pair (i, i2) of that slot, block i on waves 0-1 and block i2
// on waves 2-3, over the union of their kept lists; a wave skips the
// key blocks its own block does not keep, so each row sees exactly its own
// blocks in ascending order, as when the two run alone.
//
// F8 (the quantised-V variant): V comes as E4M3 tiles with per-channel
// power-of-two scales; the probabilities of a whole block are rounded to
// E4M3 and multiplied with one 16x16x128 fp8 MFMA per (channel tile, query
// tile), the scales entering as the MFMA's E8M0 block scales.
template <bool F8>
__device__ void process_item(const AttnParams& P, int row, int begin, int end, float* __restrict__ partial,
                             unsigned char* __restrict__ Ks, unsigned char* __restrict__ Vs, int pslot = -1,
                             int i2 = 0) {
  const int nb = P.g.nb;
  const int bh = row / nb;
  const int i = row - bh * nb;
  const int b = bh / P.heads;
  const int h = bh - b * P.heads;
  const int64_t base = (int64_t)b * P.sb + (int64_t)h * P.sh;
  const uint16_t* Qh = P.Q + base;
  const uint16_t* Kh = P.K + base;
  const uint16_t* Vh = P.V + base;
  uint16_t* Oh = P.O + base;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g4 = lane >> 4;
  const int l16 = lane & 15;
  const bool paired = pslot >= 0;
  const int half = paired ? wave >> 1 : 0;  // which block of a pair
  const int hbit = paired ? 1 << half : 0;  // this wave's skip bit in a pair's entries
  const BlockBox bi = block_box(P.g, half ? i2 : i);
  const int row0 = paired ? 32 * (wave & 1) : 32 * wave;
  const bool active = row0 < bi.n;

  // FP8 variant: the head's E4M3 V tiles, and the E8M0 scale 127 + e_d of
  // each of the lane's channels d = 16mt + l16, one byte each, four per
  // register (extracted per use: the MFMA takes a scale register whose
  // upper bytes are zero).
  const unsigned char* V8h = nullptr;
  int scv[2] = {0, 0};
  if constexpr (F8) {
    V8h = P.V8 + (int64_t)bh * nb * kV8TileBytes;
    const int32_t* ve = P.vexp + (int64_t)bh * 128 + l16;
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) {
      const int sc = min(max(127 + ve[16 * mt], 0), 254);
      scv[mt >> 2] |= sc << (8 * (mt & 3));
    }
  }

  // counts and kv_idx are read through the scalar cache (constant address
  // space: the kernel never writes them). They come from the caller: clamp
  // so a bad list cannot address outside the tensors.
  // A pair's list entries carry its skip bits from bit 16 on; kv_idx entries
  // are block ids (< nb <= 1024), and only the bits below 16 are read as one.
  typedef __attribute__((address_space(4))) const int32_t const_i32;
  const const_i32* kvl;
  int cnt;
  if (paired) {
    kvl = (const const_i32*)(P.plist + (int64_t)pslot * nb);
    cnt = min(max(((const const_i32*)P.pcount)[pslot], 0), nb);
  } else {
    const int full = min(max(((const const_i32*)P.counts)[row], 0), nb);
    begin = min(max(begin, 0), full);
    end = min(max(end, begin), full);
    kvl = (const const_i32*)(P.kv_idx + (int64_t)row * nb + begin);
    cnt = end - begin;
  }

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
        qf[nt][ks] = *reinterpret_cast<const bf16x8*>(Qh + (uint32_t)(qtok[nt] * (int)P.sn + 32 * ks + 8 * g4));
      } else {
        qf[nt][ks] = bf16x8{};
      }
    }
  }

  // Q is in registers before any tile copy is issued (a wait the compiler
  // sees, so it never re-waits for Q behind the copies).
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0), expcnt/lgkmcnt unconstrained

  f32x4 o[8][2];
#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) o[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrow[2] = {-1.0e30f, -1.0e30f};
  // Per row, the score above which the reference moves (mrow + 8 / c2 for
  // bf16 P, mrow + 1 / c2 for E4M3 P) and the exponent offset (-mrow * c2,
  // plus 7 for E4M3 P), both refreshed only when mrow moves.
  const float move_ref = (F8 ? 1.0f : 8.0f) / P.c2;
  constexpr float kPOffset = F8 ? 7.0f : 0.0f;
  float thr[2] = {-1.0e30f, -1.0e30f};
  float negm[2] = {0.f, 0.f};
  // Softmax denominators on the matrix unit: an extra O^T tile whose V^T
  // operand is all ones accumulates sum_k P[k] for every query row (all 16
  // rows of the tile hold it), rescaled together with O.
  f32x4 lsum[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  bf16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = (__bf16)1.0f;

  // Lane constants of the transposing V reads: source lane 4e + q of group g4
  // points at row 32kg + 16hf + 4g4 + e, 8-byte chunk 4mt + q (swizzled).
  const int te = l16 >> 2;
  const int tq = l16 & 3;
  const int vrow = (4 * g4 + te) * kRowBytes;
  const int vsw = (4 * g4 + te) & 7;

  // The kept-block id and block record of the next block are fetched one
  // block ahead (during the current block's softmax), so their scalar loads
  // never stall the copy of the next tiles.
  int roff[8];
  const int e0 = cnt > 0 ? kvl[0] : 0;
  const int e1 = cnt > 1 ? kvl[1] : 0;
  const int jc = min(e0 & 0xFFFF, nb - 1);
  BlockMap mc = load_block_map(P.bmap, jc);
  int j1 = min(e1 & 0xFFFF, nb - 1);
  // skip bits of the current block (bits 0-1) and of the next (bits 2-3)
  int fq = ((e0 >> 16) & 3) | (((e1 >> 16) & 3) << 2);
  if (cnt > 0) {
    row_offsets(P, mc, roff);
    if (wave < ngroups_of(mc.n)) {
      issue_tile<false>(Kh, roff, Ks);
      if constexpr (!F8) issue_tile<true>(Vh, roff, Vs);
    }
    if constexpr (F8) issue_v8_tile(V8h, jc, Vs);
  }

  // LDS addresses of the lane's fragments, formed once per item: the
  // swizzled lane part differs per V channel tile mt and per K head-dim step
  // ks, and the rest (key group, K row tile) is an immediate offset. In the
  // bf16 kernel they are opaque to the compiler, which would otherwise
  // re-add the lane parts at every read.
  uint32_t vaddr[8], kaddr[4];
  {
    const uint32_t vbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)Vs;
    const uint32_t kbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)Ks;
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) vaddr[mt] = vbase + (uint32_t)(vrow + 8 * (4 * (mt ^ vsw) + tq));
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) kaddr[ks] = kbase + (uint32_t)(l16 * kRowBytes + 16 * ((4 * ks + g4) ^ l16));
    if constexpr (!F8) {  // (the FP8 kernel has no registers to spare for them)
      asm volatile("" : "+v"(vaddr[0]), "+v"(vaddr[1]), "+v"(vaddr[2]), "+v"(vaddr[3]), "+v"(vaddr[4]),
                   "+v"(vaddr[5]), "+v"(vaddr[6]), "+v"(vaddr[7]));
      asm volatile("" : "+v"(kaddr[0]), "+v"(kaddr[1]), "+v"(kaddr[2]), "+v"(kaddr[3]));
    }
  }
  typedef __attribute__((address_space(3))) unsigned char lds_u8;
  typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
  auto vfrag = [&](int kg, int mt) {
    lds_u8* vb = (lds_u8*)(uintptr_t)vaddr[mt] + kg * 32 * kRowBytes;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)vb);
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vb + 16 * kRowBytes));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  auto kfrag = [&](int mt, int ks) {
    return *(lds_bf16x8*)((lds_u8*)(uintptr_t)kaddr[ks] + mt * 16 * kRowBytes);
  };

  // One half of a block: S^T for its key groups (LDS tiles 4hb .. 4hb + 3),
  // the online softmax, and the PV product. A short half (the second half of
  // a block with 65 .. 96 keys) has only its first group of 32 keys: the
  // steps of the second group are skipped by uniform branches, so there is
  // one code path for both shapes. The K (V) fragment of step u + 2 is read
  // while step u multiplies (a ring of three fragments), so the LDS latency
  // is covered by four MFMAs.
  auto s_phase = [&](int hb, bool short_half, f32x4 (&s)[4][2]) {
    constexpr int kKPre = 2;
    bf16x8 kq[kKPre + 1];
#pragma unroll
    for (int u = 0; u < kKPre; ++u) kq[u] = kfrag(4 * hb + 2 * (u >> 3) + (u & 1), (u & 7) >> 1);
    // Issue priority while multiplying: the SIMD's other wave (another
    // workgroup, usually in its softmax) fills the matrix unit's gaps.
    __builtin_amdgcn_s_setprio(2);
    // Step u of a group of eight (u / 8 = pair of 16-key tiles) takes tile
    // 2 (u / 8) + u % 2 at head-dim step (u % 8) / 2: four independent
    // accumulation chains (two tiles x two query tiles) alternate, so a
    // dependent product never follows its predecessor directly.
    auto t_of = [](int u) { return 2 * (u >> 3) + (u & 1); };
    auto ks_of = [](int u) { return (u & 7) >> 1; };
    auto step = [&](auto u_c) {
      constexpr int u = decltype(u_c)::value;
      constexpr int t = 2 * (u >> 3) + (u & 1), ks = (u & 7) >> 1;
      if (u + kKPre < 16) kq[(u + kKPre) % (kKPre + 1)] = kfrag(4 * hb + t_of(u + kKPre), ks_of(u + kKPre));
      const bf16x8 ka = kq[u % (kKPre + 1)];
      const f32x4 z = f32x4{0.f, 0.f, 0.f, 0.f};
      s[t][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[0][ks], ks == 0 ? z : s[t][0], 0, 0, 0);
      s[t][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[1][ks], ks == 0 ? z : s[t][1], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    };
    static_for<0, 8>(step);
    if (!short_half) static_for<8, 16>(step);
    __builtin_amdgcn_s_setprio(0);
  };

  // Online softmax over the half. Accumulator (t, r) of lane group g4 holds
  // key 64hb + 32*(t/2) + 8*g4 + 4*(t%2) + r; keys past nj are masked (in a
  // short half that covers every key of tiles 2 and 3).
  auto softmax_phase = [&](int hb, bool short_half, int nj, f32x4 (&s)[4][2], bf16x8 (&pb)[2][2]) {
    if (nj < 64 * hb + 64) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kap = 64 * hb + 32 * (t >> 1) + 8 * g4 + 4 * (t & 1) + r;
          if (kap >= nj) {
            s[t][0][r] = -INFINITY;
            s[t][1][r] = -INFINITY;
          }
        }
      }
    }
    float mx[2] = {-INFINITY, -INFINITY};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        mx[0] = fmaxf(mx[0], s[t][0][r]);
        mx[1] = fmaxf(mx[1], s[t][1][r]);
      }
    }
    // The exponent reference mrow only moves when a row's max exceeds it
    // by more than 2^8 (in exp2 units): P stays <= 256, exact in bf16
    // scaling, and the O rescale is rare. O and l share the reference, so
    // the final O / l is unchanged. A row's max is the max over its four
    // lane groups, all in this wave: when no lane's own max passes the
    // threshold, no row's does, and the cross-lane max is skipped.
    if (__ballot(mx[0] > thr[0] || mx[1] > thr[1])) {
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const float rmx = row_max4(mx[nt]);
        const bool grow = rmx > thr[nt];
        const float mref = grow ? rmx : mrow[nt];
        const float alpha = grow ? __builtin_amdgcn_exp2f((mrow[nt] - mref) * P.c2) : 1.0f;
        mrow[nt] = mref;
        if (__ballot(grow)) {
#pragma unroll
          for (int mt = 0; mt < 8; ++mt) o[mt][nt] *= alpha;
          lsum[nt] *= alpha;
          thr[nt] = mrow[nt] + move_ref;
          negm[nt] = -mrow[nt] * P.c2;
        }
      }
    }
    // The first 32 keys only: the exponentials of the second 32 are taken
    // inside the PV phase, under the products of the first.
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) s[t][nt][r] = __builtin_amdgcn_exp2f(fmaf(s[t][nt][r], P.c2, negm[nt]));
      }
    }
    pb[0][0] = to_bf16x8(s[0][0], s[1][0]);
    pb[0][1] = to_bf16x8(s[0][1], s[1][1]);
    (void)short_half;
  };

  // O^T += V^T P^T, 32 keys per MFMA; V^T comes from row-major V through
  // transposing LDS reads. Step u = 8kk + mt. Steps 0..7 (the first 32 keys)
  // also take the exponentials of the second 32 keys, two values a step, so
  // that VALU work runs while the matrix unit multiplies.
  auto pv_phase = [&](int hb, bool short_half, bf16x8 (&pb)[2][2], f32x4 (&s)[4][2], const float (&negm)[2]) {
    constexpr int kVPre = 2;
    bf16x8 vq[kVPre + 1];
#pragma unroll
    for (int u = 0; u < kVPre; ++u) vq[u] = vfrag(2 * hb + (u >> 3), u & 7);
    __builtin_amdgcn_s_setprio(1);
    auto step = [&](auto u_c) {
      constexpr int u = decltype(u_c)::value;
      constexpr int kk = u >> 3, mt = u & 7;
      if (u + kVPre < 16) vq[(u + kVPre) % (kVPre + 1)] = vfrag(2 * hb + ((u + kVPre) >> 3), (u + kVPre) & 7);
      const bf16x8 va = vq[u % (kVPre + 1)];
      o[mt][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb[kk][0], o[mt][0], 0, 0, 0);
      o[mt][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb[kk][1], o[mt][1], 0, 0, 0);
      if (mt == 7) {
        lsum[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[kk][0], lsum[0], 0, 0, 0);
        lsum[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[kk][1], lsum[1], 0, 0, 0);
      }
      if constexpr (u < 8) {
        // values 2u, 2u + 1 of the second group: tile 2 + u / 4, row u % 4, both query tiles
        if (!short_half) {
          constexpr int t = 2 + (u >> 2), r = u & 3;
          s[t][0][r] = __builtin_amdgcn_exp2f(fmaf(s[t][0][r], P.c2, negm[0]));
          s[t][1][r] = __builtin_amdgcn_exp2f(fmaf(s[t][1][r], P.c2, negm[1]));
        }
        if constexpr (u == 7) {
          if (!short_half) {
            pb[1][0] = to_bf16x8(s[2][0], s[3][0]);
            pb[1][1] = to_bf16x8(s[2][1], s[3][1]);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    static_for<0, 8>(step);
    if (!short_half) static_for<8, 16>(step);
    __builtin_amdgcn_s_setprio(0);
  };

  // ---- FP8 variant ------------------------------------------------------
  // E4M3 V^T fragment of channel tile mt: lane (g4, l16) holds channel
  // 16mt + l16, key positions 32g4 .. 32g4 + 31 (two 16-byte chunks, stored
  // at physical chunk (logical ^ (channel % 8))).
  const int v8o0 = l16 * 128 + 16 * ((2 * g4) ^ (l16 & 7));
  const int v8o1 = l16 * 128 + 16 * ((2 * g4 + 1) ^ (l16 & 7));
  auto v8frag = [&](int mt) {
    const i32x4 lo = *reinterpret_cast<const i32x4*>(Vs + mt * 2048 + v8o0);
    const i32x4 hi = *reinterpret_cast<const i32x4*>(Vs + mt * 2048 + v8o1);
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  // O^T += V^T P^T over the whole block, one 16x16x128 fp8 MFMA per (channel
  // tile, query tile). A scale: 127 + e_d, the channel's V exponent; B
  // scale: 2^-7 (P was rounded as P * 2^7), times 2^-kb on the first half's
  // keys when the second half moved the row's reference (sbv). The sum of P
  // comes from the same MFMA against E4M3 ones.
  //
  // K order of the instruction: lane group g holds K = 16g .. 16g + 15 in its
  // bytes 0..15 and K = 64 + 16g .. in its bytes 16..31, and the E8M0 scale of
  // K block b (K = 32b .. 32b + 31) is lane group b's. Bytes 0..15 of every
  // group are the first half's keys (words 0..3), so the first half is K
  // blocks 0 and 1 (scales of lane groups 0 and 1), the second half K blocks
  // 2 and 3.
  auto pv_f8 = [&](const i32x8 (&p8)[2], const int (&sbv)[2]) {
    constexpr int kPre = 2;
    i32x8 vq[kPre + 1];
#pragma unroll
    for (int u = 0; u < kPre; ++u) vq[u] = v8frag(u);
    __builtin_amdgcn_s_setprio(1);
    auto step = [&](auto mt_c) {
      constexpr int mt = decltype(mt_c)::value;
      if constexpr (mt + kPre < 8) vq[(mt + kPre) % (kPre + 1)] = v8frag(mt + kPre);
      const i32x8 va = vq[mt % (kPre + 1)];
      const int sa = (scv[mt >> 2] >> (8 * (mt & 3))) & 0xFF;
      o[mt][0] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(va, p8[0], o[mt][0], 0, 0, 0, sa, 0, sbv[0]);
      o[mt][1] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(va, p8[1], o[mt][1], 0, 0, 0, sa, 0, sbv[1]);
      __builtin_amdgcn_sched_barrier(0);
    };
    static_for<0, 8>(step);
    const i32x8 ones8 = {0x38383838, 0x38383838, 0x38383838, 0x38383838,
                         0x38383838, 0x38383838, 0x38383838, 0x38383838};
    lsum[0] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ones8, p8[0], lsum[0], 0, 0, 0, 127, 0, sbv[0]);
    lsum[1] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ones8, p8[1], lsum[1], 0, 0, 0, 127, 0, sbv[1]);
    __builtin_amdgcn_s_setprio(0);
  };
  // Online softmax of one half into E4M3: accumulator (t, r) of lane group
  // g4 becomes byte r of word 4hb + t of the B operand (the order of the
  // E4M3 V tiles). The reference moves when a row's max
  // passes it by more than 1 (exp2 units), so P * 2^7 <= 2^8 stays inside the
  // format (largest finite 448) and the smallest nonzero E4M3 value sits
  // 2^-16 .. 2^-17 below the row's largest P. In the first half the move is
  // free; in the second it is a whole number kb of powers of two, so the
  // first half (already rounded against the old reference) is rescaled
  // exactly through its K blocks' MFMA scale, and O and the sum of P by 2^-kb.
  auto softmax_f8 = [&](int hb, bool short_half, int nj, f32x4 (&s)[4][2], i32x8 (&p8)[2], int (&kb)[2]) {
    if (nj < 64 * hb + 64) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kap = 64 * hb + 32 * (t >> 1) + 8 * g4 + 4 * (t & 1) + r;
          if (kap >= nj) {
            s[t][0][r] = -INFINITY;
            s[t][1][r] = -INFINITY;
          }
        }
      }
    }
    float mx[2] = {-INFINITY, -INFINITY};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        mx[0] = fmaxf(mx[0], s[t][0][r]);
        mx[1] = fmaxf(mx[1], s[t][1][r]);
      }
    }
    if (__ballot(mx[0] > thr[0] || mx[1] > thr[1])) {
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const float rmx = row_max4(mx[nt]);
        const bool grow = rmx > thr[nt];
        float alpha = 1.0f;
        if (hb == 0) {
          const float mref = grow ? rmx : mrow[nt];
          alpha = grow ? __builtin_amdgcn_exp2f((mrow[nt] - mref) * P.c2) : 1.0f;
          mrow[nt] = mref;
        } else if (grow) {
          // a whole number of powers of two, at least one
          const int k = max((int)ceilf((rmx - mrow[nt]) * P.c2 - 1.0f), 1);
          kb[nt] = k;
          mrow[nt] += (float)k / P.c2;
          alpha = k > 126 ? 0.0f : __uint_as_float((uint32_t)(127 - k) << 23);
        }
        if (__ballot(grow)) {
#pragma unroll
          for (int mt = 0; mt < 8; ++mt) o[mt][nt] *= alpha;
          lsum[nt] *= alpha;
          thr[nt] = mrow[nt] + move_ref;
          negm[nt] = kPOffset - mrow[nt] * P.c2;
        }
      }
    }
    auto tile = [&](auto t_c) {
      constexpr int t = decltype(t_c)::value;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        float e[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) e[r] = __builtin_amdgcn_exp2f(fmaf(s[t][nt][r], P.c2, negm[nt]));
        int w = __builtin_amdgcn_cvt_pk_fp8_f32(e[0], e[1], 0, false);
        w = __builtin_amdgcn_cvt_pk_fp8_f32(e[2], e[3], w, true);
        p8[nt][4 * hb + t] = w;
      }
    };
    static_for<0, 2>(tile);
    if (!short_half) static_for<2, 4>(tile);
  };
  if constexpr (F8) {
    for (int c = 0; c < cnt; ++c) {
      const int nj = mc.n;
      const int ng = ngroups_of(nj);
      // K_c landed (the four copies of V8_c, issued after it, may be in flight).
      wait_vmem<4>();
      tile_barrier();
      const bool act = active && !(fq & hbit);
      i32x8 p8[2] = {i32x8{0, 0, 0, 0, 0, 0, 0, 0}, i32x8{0, 0, 0, 0, 0, 0, 0, 0}};
      int kb[2] = {0, 0};
      BlockMap mn;
      int j2 = 0;
      {
        f32x4 s[4][2];
        if (act) s_phase(0, false, s);
        // record of block c + 1 and the entry of block c + 2 (clamped to the list)
        mn = load_block_map(P.bmap, j1);
        const int e2 = kvl[min(c + 2, cnt - 1)];
        j2 = min(e2 & 0xFFFF, nb - 1);
        fq = (fq >> 2) | (((e2 >> 16) & 3) << 2);
        if (act) softmax_f8(0, false, nj, s, p8, kb);
      }
      {
        const bool run = ng > 2;
        const bool short_half = ng == 3;
        f32x4 s[4][2];
        if (act && run) s_phase(1, short_half, s);
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the prefetched scalars
        wait_vmem<0>();                        // V8_c landed
        tile_barrier();                        // every wave is done with K_c and sees V8_c
        if (c + 1 < cnt) {
          mc = mn;
          if (wave < ngroups_of(mc.n)) {
            row_offsets(P, mc, roff);
            issue_tile<false>(Kh, roff, Ks);
          }
        }
        if (act && run) softmax_f8(1, short_half, nj, s, p8, kb);
      }
      if (act) {
        // B scale of the K block whose scale this lane supplies: lane groups
        // 0 and 1 scale the first half's keys, which carry the second half's
        // reference move
        const int sbv[2] = {g4 >= 2 ? 120 : max(120 - kb[0], 0), g4 >= 2 ? 120 : max(120 - kb[1], 0)};
        pv_f8(p8, sbv);
      }
      tile_barrier();  // every wave is done with V8_c
      if (c + 1 < cnt) issue_v8_tile(V8h, j1, Vs);
      j1 = j2;
    }
  } else {
  for (int c = 0; c < cnt; ++c) {
    const int nj = mc.n;
    const int ng = ngroups_of(nj);
    // K_c landed (V_c, issued after it, may still be in flight).
    if (wave < ng) wait_vmem<8>(); else wait_vmem<0>();
    tile_barrier();

    const bool act = active && !(fq & hbit);
    int ng_next = 0;
    BlockMap mn;
    int j2 = 0;
    // Each block is taken as two halves of 64 keys (key groups 2hb, 2hb+1):
    // S half -> online softmax -> PV half. Half 1 holds ng - 2 groups.
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
      const bool run = hb == 0 || ng > 2;
      const bool short_half = hb == 1 && ng == 3;
      f32x4 s[4][2];
      bf16x8 pb[2][2];
      if (act && run) s_phase(hb, short_half, s);
      if (hb == 0) {
        // record of block c + 1 and the entry of block c + 2 (clamped to the list)
        mn = load_block_map(P.bmap, j1);
        const int e2 = kvl[min(c + 2, cnt - 1)];
        j2 = min(e2 & 0xFFFF, nb - 1);
        fq = (fq >> 2) | (((e2 >> 16) & 3) << 2);
      }
      if (hb == 1) {
        tile_barrier();  // every wave is done with K_c
        // Next block's K streams in while this block finishes.
        if (c + 1 < cnt) {
          mc = mn;
          ng_next = ngroups_of(mc.n);
          if (wave < ng_next) {
            row_offsets(P, mc, roff);
            issue_tile<false>(Kh, roff, Ks);
          }
        }
      }
      if (act && run) softmax_phase(hb, short_half, nj, s, pb);
      if (hb == 0) {
        // The prefetched scalars have landed long ago; waiting for them here,
        // where no LDS read is in flight, keeps the PV fragment waits exact.
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
        // V_c landed: nothing was issued after it yet.
        wait_vmem<0>();
        tile_barrier();
      }
      if (act && run) pv_phase(hb, short_half, pb, s, negm);
    }
    tile_barrier();  // every wave is done with V_c
    if (c + 1 < cnt && wave < ng_next) issue_tile<true>(Vh, roff, Vs);
    j1 = j2;
  }
  }

  // Epilogue: O^T accumulator (mt, r) of lane (g4, l16) is head dim
  // 16mt + 4g4 + r of query row 16nt + l16.
  if (active && partial) {
    // chunk of a split row: O^T as is, the reference and the sum of P
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int r = row0 + 16 * nt + l16;
      if (r < bi.n) {
        float* prow = partial + r * 128 + 4 * g4;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) *reinterpret_cast<f32x4*>(prow + 16 * mt) = o[mt][nt];
        if (g4 == 0) {
          partial[128 * 128 + r] = mrow[nt];
          partial[128 * 128 + 128 + r] = lsum[nt][0];
        }
      }
    }
    return;
  }
  if (active) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      if (qtok[nt] >= 0) {
        const float inv = lsum[nt][0] > 0.f ? 1.0f / lsum[nt][0] : 0.f;
        uint16_t* orow = Oh + (uint32_t)(qtok[nt] * (int)P.sn + 4 * g4);
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) {
          const f32x4 v = o[mt][nt] * inv;
          *reinterpret_cast<bf16x4*>(orow + 16 * mt) = __builtin_convertvector(v, bf16x4);
        }
      }
    }
  }
}

// Trace record r: rows first, then chunk items (chunk c at n_rows + c):
// start and end on the 100 MHz constant clock, where the item ran, and the
// shader-clock cycles (s_memtime) it took, so that the engine clock of the
// run is the ratio of the two clocks. A pair's item fills the records of
// both its rows, splitting its time evenly between them. One thread writes.
__device__ __forceinline__ void trace_record(const AttnParams& P, int64_t rec, int poff, int64_t t0, int64_t t1,
                                             int64_t cycles) {
  const int64_t loc = (int64_t)hw_location();
  int64_t* tr = P.trace + rec * 4;
  if (poff) {  // a pair: the second row's record is poff records on
    const int64_t tm = t0 + (t1 - t0) / 2;
    const int64_t cm = cycles / 2;
    int64_t* t2 = tr + 4 * (int64_t)poff;
    tr[0] = t0;
    tr[1] = tm;
    tr[2] = loc;
    tr[3] = cm;
    t2[0] = tm;
    t2[1] = t1;
    t2[2] = loc;
    t2[3] = cycles - cm;
  } else {
    tr[0] = t0;
    tr[1] = t1;
    tr[2] = loc;
    tr[3] = cycles;
  }
}

template <bool F8>
__global__ __launch_bounds__(kAttnThreads, 2) void attn_naive_kernel(AttnParams P) {
  __shared__ __align__(16) unsigned char ks_tile[kTileBytes];
  __shared__ __align__(16) unsigned char vs_tile[F8 ? kV8TileBytes : kTileBytes];
  const int64_t t0 = (int64_t)wall_clock64();
  const int64_t c0 = P.trace ? (int64_t)__builtin_amdgcn_s_memtime() : 0;
  process_item<F8>(P, blockIdx.x, 0, P.g.nb, nullptr, ks_tile, vs_tile);
  if (P.trace) {
    __syncthreads();
    if (threadIdx.x == 0) {
      const int64_t c1 = (int64_t)__builtin_amdgcn_s_memtime();
      trace_record(P, blockIdx.x, 0, t0, (int64_t)wall_clock64(), c1 - c0);
    }
  }
}

// Persistent scheduler. The work list holds kQueues queues, one per XCD;
// workgroups pull from the queue of the XCD they run on and steal from the
// others once theirs is empty.
constexpr int kQueues = 8;

// Role of row r (= bh * nb + i) under query-block pairing with chunk size S:
// 1 when it starts a pair (its item runs row r and its partner's row), 2
// when it is the second row of a pair (its item does nothing), 0 otherwise.
// A pair is formed only when neither row is split (kept count <= S). The
// persistent kernel decides it with this function, from the block records'
// partner offsets; the plan and the pair-list kernel apply the same test.
__device__ __forceinline__ int pair_role(const BlockMap* __restrict__ table, const int32_t* __restrict__ counts,
                                         int r, int i, int S, int nb) {
  auto whole = [&](int rr) { return min(max(counts[rr], 0), nb) <= S; };
  const int poff = table[i].poff;
  if (poff == 0 || !whole(r) || !whole(r + poff)) return 0;
  return poff > 0 ? 1 : 2;
}

__device__ __forceinline__ int xcc_id() {
  uint32_t xcc;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
  return (int)(xcc & 0xfu);
}

template <bool F8>
__global__ __launch_bounds__(kAttnThreads, 2) void attn_persistent_kernel(AttnParams P, const int32_t* __restrict__ items,
                                                                          const int32_t* __restrict__ qbase,
                                                                          int32_t* __restrict__ qctr) {
  __shared__ __align__(16) unsigned char ks_tile[kTileBytes];
  __shared__ __align__(16) unsigned char vs_tile[F8 ? kV8TileBytes : kTileBytes];
  __shared__ int next_slot, next_q;
  int q = xcc_id() % kQueues;
  // The trace record of an item is written at the top of the next iteration,
  // by thread 0 together with the queue pop: the loop then holds a single
  // region that only thread 0 runs, so the compiler keeps every lane of
  // every wave on one path through the loop and its barriers.
  int64_t prec = -1, pt0 = 0, pt1 = 0, pcyc = 0;
  int ppoff = 0;
  for (;;) {
    if (threadIdx.x == 0) {
      if (prec >= 0) trace_record(P, prec, ppoff, pt0, pt1, pcyc);
      int slot = -1, qq = q;
      for (int t = 0; t < kQueues; ++t) {
        qq = (q + t) % kQueues;
        const int len = qbase[qq + 1] - qbase[qq];
        if (len <= 0) continue;
        const int k = atomicAdd(&qctr[qq], 1);
        if (k < len) {
          slot = qbase[qq] + k;
          break;
        }
      }
      next_slot = slot;
      next_q = qq;
    }
    __syncthreads();
    const int slot = __builtin_amdgcn_readfirstlane(next_slot);
    q = __builtin_amdgcn_readfirstlane(next_q);  // keep stealing from a queue that had work
    if (slot < 0) break;
    // item >= 0: a whole row; item < 0: chunk -1 - item of a split row
    const int item = __builtin_amdgcn_readfirstlane(items[slot]);
    const int64_t t0 = (int64_t)wall_clock64();
    const int64_t c0 = P.trace ? (int64_t)__builtin_amdgcn_s_memtime() : 0;
    // One call site for every kind of item (rows, pairs, chunks), so that the
    // item body is inlined once.
    int row = item, begin = 0, end = P.g.nb, pslot = -1, poff = 0, i2 = 0;
    float* partial = nullptr;
    int64_t rec = item;
    if (item >= 0) {
      const int bh = item / P.g.nb;
      const int i = item - bh * P.g.nb;
      const int role = P.plist ? pair_role(P.bmap, P.counts, item, i, *P.psplit, P.g.nb) : 0;
      if (role == 1) {
        pslot = bh * P.pairs_head + P.bmap[i].pslot;
        poff = P.bmap[i].poff;
        i2 = i + poff;
      }
      rec = role == 2 ? -1 : item;  // the pair's item records the second row
    } else {
      const int c = -1 - item;
      typedef __attribute__((address_space(4))) const int32_t const_i32;
      const const_i32* ch = (const const_i32*)(P.chunks + c);
      row = ch[0];
      begin = ch[1];
      end = ch[2];
      partial = P.partials + (int64_t)c * kPartialFloats;
      rec = c < P.trace_chunks ? P.n_rows + c : -2;
    }
    if (rec != -1) process_item<F8>(P, row, begin, end, partial, ks_tile, vs_tile, pslot, i2);
    __syncthreads();  // the next item's copies overwrite the tiles; next_slot is rewritten
    if (P.trace) {
      prec = rec;
      ppoff = poff;
      pt0 = t0;
      pt1 = (int64_t)wall_clock64();
      pcyc = (int64_t)__builtin_amdgcn_s_memtime() - c0;
    }
  }
}

constexpr int kMinChunk = 32;      // smallest automatic chunk (kept blocks)
constexpr int kPlanLdsHeads = 1024;  // heads whose queue bookkeeping the plan keeps in LDS

// Builds the work list (one workgroup of 1024 threads).
//
// Chunks (the split part of the scheduler): with S = `forced` (> 0) or, by
// default, S = max(kMinChunk, ceil(total / (2 * slots))), total being the sum
// over rows of (kept blocks + 1), a row keeping more than S blocks becomes
// ceil(count / S) chunk items of nearly equal length, each a separate work
// item whose partial result combine_kernel merges. The default S splits only
// rows longer than about half a workgroup slot's fair share, so with many
// rows per slot nothing is split; it also bounds the chunks by 4 * slots
// (the sum of ceil(c / S) over rows with c > S is at most 2 * total / S). If
// the chunks would exceed chunk_cap, no row is split.
//
// Pairs (pairing != 0): the final S goes to *psplit for the pair-list and
// attention kernels; a pair's first row costs its larger kept count + 1 (the
// union it runs is about that long) and its second row 1 (an empty item).
//
// Queues: heads are taken in decreasing order of cost. Each head's query
// blocks are cut into kQueues contiguous runs of about equal cost, run x going
// to queue x (the items of a split row stay together), so all XCDs work on the
// same head at the same time (its K/V stay in the shared last-level cache)
// and the resident workgroups of one XCD work on neighbouring query blocks
// (their kept K/V blocks overlap in L2).
//
// Scratch: per head cost, rank, run starts [kQueues + 1], queue offsets
// [kQueues]; per row the exclusive prefixes of chunks and split rows.
__global__ __launch_bounds__(1024) void plan_kernel(const int32_t* __restrict__ counts, int n_heads, Geometry g,
                                                   int slots, int forced, int chunk_cap, int32_t* __restrict__ items,
                                                   int32_t* __restrict__ qbase, int32_t* __restrict__ qctr,
                                                   int32_t* __restrict__ hscratch, int32_t* __restrict__ rscratch,
                                                   int4* __restrict__ chunks, int4* __restrict__ splits,
                                                   int32_t* __restrict__ n_split, const BlockMap* __restrict__ table,
                                                   int pairing, int32_t* __restrict__ psplit) {
  __shared__ long long wtot[16];
  __shared__ int lds_order[kPlanLdsHeads];
  __shared__ int lds_cost[kPlanLdsHeads];
  __shared__ int lds_len[kPlanLdsHeads * kQueues];
  __shared__ int poffs[kMaxBlocks];
  const int nb = g.nb;
  const int rows = n_heads * nb;
  const bool in_lds = n_heads <= kPlanLdsHeads;
  int32_t* hcost = hscratch;
  int32_t* horder = hcost + n_heads;
  int32_t* hstart = horder + n_heads;                  // [n_heads][kQueues + 1]
  int32_t* hoff = hstart + (size_t)n_heads * (kQueues + 1);  // [n_heads][kQueues]
  int32_t* cpre = rscratch;                            // [rows + 1] chunks before row r
  int32_t* spre = cpre + rows + 1;                     // [rows + 1] split rows before row r
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  auto kept_of = [&](int r) {
    const int c = counts[r];
    return c < 0 ? 0 : (c > nb ? nb : c);
  };

  // 0. chunk size. One workgroup does all of the plan, so its time is load
  //    latency: every thread keeps eight loads in flight per step (lanes past
  //    the last row re-read it), here and in the passes below.
  long long tsum = 0;
  for (int r0 = threadIdx.x; r0 < rows; r0 += 8 * (int)blockDim.x) {
    int c8[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) c8[u] = counts[min((int64_t)r0 + (int64_t)u * blockDim.x, (int64_t)rows - 1)];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int c = c8[u] < 0 ? 0 : (c8[u] > nb ? nb : c8[u]);
      tsum += (int64_t)r0 + (int64_t)u * blockDim.x < rows ? c + 1 : 0;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) tsum += __shfl_xor(tsum, o);
  if (lane == 0) wtot[wave] = tsum;
  __syncthreads();
  long long total = 0;
  for (int w = 0; w < nwaves; ++w) total += wtot[w];
  __syncthreads();  // wtot is reused below; every wave holds the same total
  int S = forced > 0 ? forced : (int)max((long long)kMinChunk, (total + 2LL * slots - 1) / (2LL * slots));

  // 1. items per row (1, or its chunks): when no row can exceed S (the usual
  //    case with many rows per slot) item r is row r and nothing else is
  //    built. Otherwise one pass over tiles of 1024 rows scans, packed in one
  //    64-bit word, the chunks (low half) and split rows (high half) before
  //    every row; the items before row r are r + chunks - split rows.
  const bool may_split = S < nb;
  if (may_split) {
    for (int attempt = 0; attempt < 2; ++attempt) {
      auto packed = [&](int r) -> uint64_t {
        if (r >= rows) return 0ull;
        const int c = kept_of(r);
        return c > S ? ((uint64_t)1 << 32) | (uint64_t)((c + S - 1) / S) : 0ull;
      };
      uint64_t run = 0;  // over the tiles before this one
      for (int base = 0; base < rows; base += 1024) {
        const int r = base + (int)threadIdx.x;
        const uint64_t v = packed(r);
        const uint64_t incl = wave_incl_scan_u64(v, lane);
        if (lane == 63) wtot[wave] = (long long)incl;
        __syncthreads();
        uint64_t before = run, all = run;
        for (int w = 0; w < nwaves; ++w) {
          const uint64_t t = (uint64_t)wtot[w];
          before += w < wave ? t : 0ull;
          all += t;
        }
        __syncthreads();
        if (r < rows) {
          const uint64_t ex = before + incl - v;
          cpre[r] = (int)(uint32_t)ex;
          spre[r] = (int)(ex >> 32);
        }
        run = all;
      }
      if ((int)(uint32_t)run > chunk_cap && attempt == 0) {
        S = 0x7fffffff;  // nothing is split
        continue;
      }
      if (threadIdx.x == 0) {
        cpre[rows] = (int)(uint32_t)run;
        spre[rows] = (int)(run >> 32);
        *n_split = (int)(run >> 32);
      }
      break;
    }
  } else if (threadIdx.x == 0) {
    *n_split = 0;
  }
  __syncthreads();
  // items before row r (ipre[r])
  auto ipre = [&](int r) { return may_split ? r + cpre[r] - spre[r] : r; };
  if (pairing && threadIdx.x == 0) *psplit = S;
  // Pair partner offset of every block (> 0: first of a pair, < 0: second,
  // 0: none), from the block records once; the same rule as pair_role.
  for (int i = threadIdx.x; i < nb; i += blockDim.x) poffs[i] = pairing ? table[i].poff : 0;
  __syncthreads();
  // cost of a row from its partner offset, its kept count and its partner's
  auto row_cost = [&](int poff, int c, int cn) {
    if (poff == 0 || c > S || cn > S) return c + 1;  // not in a formed pair
    return poff > 0 ? max(c, cn) + 1 : 1;
  };
  auto clamp_count = [&](int c) { return c < 0 ? 0 : (c > nb ? nb : c); };

  // 2. head costs and equal-cost runs (one wave per head): every count the
  //    head's costs need is loaded first (lanes past nb re-read the last
  //    block's; an unpaired row reads its own count as its partner's); a
  //    lane's costs stay in registers between the two passes
  for (int h = wave; h < n_heads; h += nwaves) {
    const int32_t* hc = counts + (size_t)h * nb;
    int pf[kMaxBlocks / 64], ca[kMaxBlocks / 64], cb[kMaxBlocks / 64];
#pragma unroll
    for (int k = 0; k < kMaxBlocks / 64; ++k) pf[k] = poffs[min(64 * k + lane, nb - 1)];
#pragma unroll
    for (int k = 0; k < kMaxBlocks / 64; ++k) {
      const int i = min(64 * k + lane, nb - 1);
      ca[k] = hc[i];
      cb[k] = hc[i + pf[k]];
    }
    int cst[kMaxBlocks / 64];
    int hsum = 0;
#pragma unroll
    for (int k = 0; k < kMaxBlocks / 64; ++k) {
      const int cost = row_cost(pf[k], clamp_count(ca[k]), clamp_count(cb[k]));
      cst[k] = 64 * k + lane < nb ? cost : 0;
      hsum += cst[k];
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) hsum += __shfl_xor(hsum, o);
    if (lane == 0) {
      hcost[h] = hsum;
      if (in_lds) lds_cost[h] = hsum;
    }
    // run of row i = floor(kQueues * (cost before row i) / hsum), a
    // non-decreasing function of i; run x starts at the first row whose run
    // is >= x (nb when there is none).
    int stx[kQueues + 1];
#pragma unroll
    for (int x = 0; x <= kQueues; ++x) stx[x] = nb;
    int run_before = 0;
#pragma unroll
    for (int k = 0; k < kMaxBlocks / 64; ++k) {
      const int i0 = 64 * k;
      if (i0 < nb) {  // (a guard, not a break: the loop stays unrolled and cst in registers)
        const int i = i0 + lane;
        const int c = cst[k];
        const int incl = wave_incl_scan_i32(c, lane);
        const int before = run_before + incl - c;
        // run >= x exactly when kQueues * before >= x * hsum: no division,
        // and no overflow (before <= hsum <= nb * (nb + 1))
#pragma unroll
        for (int x = 0; x < kQueues; ++x) {
          const uint64_t hit = __ballot(i < nb && before * kQueues >= x * hsum);
          if (stx[x] == nb && hit) stx[x] = i0 + __ffsll((unsigned long long)hit) - 1;
        }
        run_before += __shfl(incl, 63);
      }
    }
    int32_t* st = hstart + (size_t)h * (kQueues + 1);
    if (lane == 0) {
#pragma unroll
      for (int x = 0; x <= kQueues; ++x) st[x] = stx[x];
    }
  }
  __syncthreads();

  // 3. head order by decreasing cost (ties: lower head first), from the LDS
  //    copy of the costs when it holds them
  auto rank_by_cost = [&](const int32_t* costs, int h) {
    const int ch = costs[h];
    int rank = 0;
    for (int k = 0; k < n_heads; ++k) {
      const int ck = costs[k];
      rank += (ck > ch || (ck == ch && k < h)) ? 1 : 0;
    }
    return rank;
  };
  for (int h = threadIdx.x; h < n_heads; h += blockDim.x)
    horder[in_lds ? rank_by_cost(lds_cost, h) : rank_by_cost(hcost, h)] = h;
  __syncthreads();

  // 4. queue offsets (in items) of every (head, run) and queue bases: a
  //    walk over the heads in cost order, from LDS copies of the order and
  //    of the item count of every (head, run) when they fit
  if (in_lds) {
    for (int r = threadIdx.x; r < n_heads; r += blockDim.x) {
      const int h = horder[r];
      const int32_t* st = hstart + (size_t)h * (kQueues + 1);
      int stx[kQueues + 1], ip[kQueues + 1];
#pragma unroll
      for (int x = 0; x <= kQueues; ++x) stx[x] = st[x];
#pragma unroll
      for (int x = 0; x <= kQueues; ++x) ip[x] = ipre(h * nb + stx[x]);
      lds_order[r] = h;
#pragma unroll
      for (int x = 0; x < kQueues; ++x) lds_len[r * kQueues + x] = ip[x + 1] - ip[x];
    }
    __syncthreads();
  }
  if (threadIdx.x < kQueues) {
    const int x = threadIdx.x;
    int run = 0;
    for (int r = 0; r < n_heads; ++r) {
      int h, len;
      if (in_lds) {
        h = lds_order[r];
        len = lds_len[r * kQueues + x];
      } else {
        h = horder[r];
        const int32_t* st = hstart + (size_t)h * (kQueues + 1);
        len = ipre(h * nb + st[x + 1]) - ipre(h * nb + st[x]);
      }
      hoff[(size_t)h * kQueues + x] = run;
      run += len;
    }
    qctr[x] = run;  // queue length for now
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int base = 0;
    for (int x = 0; x < kQueues; ++x) {
      const int len = qctr[x];
      qbase[x] = base;
      base += len;
    }
    qbase[kQueues] = base;
  }
  __syncthreads();

  // 5. scatter items (a split row's chunks consecutively), chunk and split
  //    records; one wave per head, whose run x fills one contiguous slice of
  //    queue x. Then reset the queue counters.
  for (int h = wave; h < n_heads; h += nwaves) {
    // the head's run starts and the start of its slice of every queue, one
    // per lane, loaded together
    const int32_t* st = hstart + (size_t)h * (kQueues + 1);
    const int st_l = lane <= kQueues ? st[lane] : 0;
    const int off_l = lane < kQueues ? qbase[lane] + hoff[(size_t)h * kQueues + lane] : 0;
    for (int x = 0; x < kQueues; ++x) {
      const int i_begin = __builtin_amdgcn_readlane(st_l, x);
      const int i_end = __builtin_amdgcn_readlane(st_l, x + 1);
      if (i_begin >= i_end) continue;
      const int slice = __builtin_amdgcn_readlane(off_l, x) - ipre(h * nb + i_begin);
      for (int i = i_begin + lane; i < i_end; i += 64) {
        const int r = h * nb + i;
        const int pos = slice + ipre(r);
        const int n = ipre(r + 1) - ipre(r);
        if (n == 1) {
          items[pos] = r;
        } else {
          const int c0 = cpre[r];
          const int cnt = kept_of(r);
          for (int c = 0; c < n; ++c) {
            items[pos + c] = -1 - (c0 + c);
            chunks[c0 + c] = make_int4(r, (int)(((int64_t)c * cnt) / n), (int)(((int64_t)(c + 1) * cnt) / n), 0);
          }
          splits[spre[r]] = make_int4(r, c0, n, 0);
        }
      }
    }
  }
  __syncthreads();
  if (threadIdx.x < kQueues) qctr[threadIdx.x] = 0;
}

// Union lists of the query-block pairs, one wave per pair slot (pairs with a
// split row are not formed and skipped): the two rows' kept sets become bitmaps in LDS,
// read back in ascending block order as entries j | (j not kept by the first
// row) << 16 | (j not kept by the second row) << 17. An entry repeated in a
// kept list counts once.
constexpr int kPairWords = kMaxBlocks / 64;

__global__ __launch_bounds__(256) void pair_list_kernel(const int32_t* __restrict__ counts,
                                                        const int32_t* __restrict__ kv_idx, int n_heads, int nb,
                                                        const BlockMap* __restrict__ table, int pairs_head,
                                                        const int32_t* __restrict__ pfirst,
                                                        const int32_t* __restrict__ psplit, int32_t* __restrict__ plist,
                                                        int32_t* __restrict__ pcount) {
  __shared__ unsigned long long bits[4][2 * kPairWords];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int S = *psplit;
  const int n_pairs = n_heads * pairs_head;
  unsigned long long* bw = bits[wave];
  auto whole = [&](int rr) { return min(max(counts[rr], 0), nb) <= S; };
  for (int slot = blockIdx.x * 4 + wave; slot < n_pairs; slot += gridDim.x * 4) {
    const int bh = slot / pairs_head;
    const int i = pfirst[slot - bh * pairs_head];
    const int r = bh * nb + i;
    const int r2 = r + table[i].poff;
    if (!whole(r) || !whole(r2)) continue;  // not formed: both rows run alone
    if (lane < 2 * kPairWords) bw[lane] = 0ull;
    wave_sync();
    for (int s = 0; s < 2; ++s) {
      const int rs = s ? r2 : r;
      const int c = min(max(counts[rs], 0), nb);
      const int32_t* kv = kv_idx + (int64_t)rs * nb;
      for (int a = lane; a < c; a += 64) {
        const int j = min(max(kv[a], 0), nb - 1);
        atomicOr(&bw[s * kPairWords + (j >> 6)], 1ull << (j & 63));
      }
    }
    wave_sync();
    int32_t* out = plist + (int64_t)slot * nb;
    int n = 0;
    for (int w = 0; w * 64 < nb; ++w) {
      const int j = 64 * w + lane;
      const int ka = (int)((bw[w] >> lane) & 1ull);
      const int kb = (int)((bw[kPairWords + w] >> lane) & 1ull);
      const bool keep = (ka | kb) != 0;  // bits past nb are never set
      const uint64_t m = __ballot(keep);
      if (keep) out[n + lanes_below(m)] = j | ((ka ^ 1) << 16) | ((kb ^ 1) << 17);
      n += __popcll(m);
    }
    if (lane == 0) pcount[slot] = n;
    wave_sync();  // the bitmaps are cleared for the next pair only after every lane read them
  }
}

// Merges the chunks of every split row (one workgroup per row at a time, in
// chunk order, so the result is deterministic): with m_c the chunk's
// exponent reference, l_c its sum of P and O_c its unnormalised output,
// O = sum_c w_c O_c / sum_c w_c l_c, w_c = exp2((m_c - max_c m_c) * c2).
// Thread t takes query row t / 2, head dims 64 (t % 2) .. +63.
__global__ __launch_bounds__(256) void combine_kernel(AttnParams P, const int4* __restrict__ splits,
                                                     const int32_t* __restrict__ n_split) {
  const int ns = __builtin_amdgcn_readfirstlane(*n_split);
  const int nb = P.g.nb;
  const int q = threadIdx.x >> 1;
  const int half = threadIdx.x & 1;
  for (int si = blockIdx.x; si < ns; si += gridDim.x) {
    const int4 sp = splits[si];
    const int row = sp.x, c0 = sp.y, n = sp.z;
    const int bh = row / nb;
    const int i = row - bh * nb;
    const int b = bh / P.heads;
    const int h = bh - b * P.heads;
    const BlockBox bi = block_box(P.g, i);
    if (q >= bi.n) continue;
    const float* part0 = P.partials + (int64_t)c0 * kPartialFloats;
    float M = -INFINITY;
    for (int c = 0; c < n; ++c) M = fmaxf(M, part0[(int64_t)c * kPartialFloats + 128 * 128 + q]);
    f32x4 acc[16];
#pragma unroll
    for (int d = 0; d < 16; ++d) acc[d] = f32x4{0.f, 0.f, 0.f, 0.f};
    float L = 0.f;
    for (int c = 0; c < n; ++c) {
      const float* pc = part0 + (int64_t)c * kPartialFloats;
      const float w = __builtin_amdgcn_exp2f((pc[128 * 128 + q] - M) * P.c2);
      L += w * pc[128 * 128 + 128 + q];
      const f32x4* src = reinterpret_cast<const f32x4*>(pc + q * 128 + 64 * half);
#pragma unroll
      for (int d = 0; d < 16; ++d) acc[d] += w * src[d];
    }
    const float inv = L > 0.f ? 1.0f / L : 0.f;
    const int64_t base = (int64_t)b * P.sb + (int64_t)h * P.sh;
    uint16_t* orow = P.O + base + (int64_t)box_token(P.g, bi, q) * P.sn + 64 * half;
#pragma unroll
    for (int d = 0; d < 16; ++d) *reinterpret_cast<bf16x4*>(orow + 4 * d) = __builtin_convertvector(acc[d] * inv, bf16x4);
  }
}

static_assert(kMaxBlocks <= 1024, "block_table_kernel runs one thread per block in one workgroup");

// Block records of every block of the tiling, one thread per block in one
// workgroup (nb <= 1024), the query-block pairs numbered in the order of
// their first block; and (pfirst != null) the first block of every pair.
__global__ __launch_bounds__(1024) void block_table_kernel(Geometry g, BlockMap* __restrict__ table,
                                                          int32_t* __restrict__ pfirst) {
  __shared__ int wsum[1024 / 64];
  const int j = threadIdx.x;
  const int lane = j & 63;
  const int wave = j >> 6;
  BlockMap m = {};
  int first = 0;
  if (j < g.nb) {
    m = block_map(g, j);
    first = m.poff > 0 ? 1 : 0;
  }
  const int incl = wave_incl_scan_i32(first, lane);
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int before = incl - first;
  for (int w = 0; w < wave; ++w) before += wsum[w];
  if (j < g.nb) {
    m.pslot = first ? before : -1;
    table[j] = m;
    if (pfirst && first) pfirst[before] = j;
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
  int per_cu = 0;    // resident workgroups of the bf16 kernel per CU
  int per_cu8 = 0;   // same for the FP8 variant
};

// Per-device occupancy, filled on a device's first call. Calls may come from
// several host threads at once: the cache is read and written under one lock.
hipError_t device_info(DeviceInfo& info) {
  static DeviceInfo cache[64];
  static std::mutex cache_lock;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> guard(cache_lock);
  if (cache[dev].cus == 0) {
    DeviceInfo d;
    e = hipDeviceGetAttribute(&d.cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &d.per_cu, reinterpret_cast<const void*>(&attn_persistent_kernel<false>), kAttnThreads, 0);
    if (e != hipSuccess) return e;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &d.per_cu8, reinterpret_cast<const void*>(&attn_persistent_kernel<true>), kAttnThreads, 0);
    if (e != hipSuccess) return e;
    if (d.per_cu < 1) d.per_cu = 1;
    if (d.per_cu8 < 1) d.per_cu8 = 1;
    cache[dev] = d;
  }
  info = cache[dev];
  return hipSuccess;
}

}  // namespace

namespace {
struct AttnWorkspace {
  int32_t* counts;   // [rows]        rebuilt counts (caller passed none)
  int32_t* kv;       // [rows][nb]    rebuilt kept lists
  int32_t* items;    // [rows + cap]  queue contents
  int32_t* qbase;    // [kQueues + 1]
  int32_t* qctr;     // [kQueues]
  int32_t* hscratch; // [heads * (2 + 2 * kQueues + 1)]
  int32_t* rscratch; // [2 * (rows + 1)] per-row prefixes
  int32_t* n_split;  // [1]
  int4* chunks;      // [cap]
  int4* splits;      // [cap]
  float* partials;   // [cap][kPartialFloats]
  BlockMap* bmap;    // [nb]
  int32_t* plist;    // [pairs][nb]   union lists of query-block pairs (null: no pairing)
  int32_t* pcount;   // [pairs]
  int32_t* pfirst;   // [pairs per head] first block of each pair slot
  int32_t* psplit;   // [1]           the plan's chunk size
  int pairs_head;    // pairs per head
  int cap;           // chunk records
  size_t bytes;
};

// The automatic chunk size assumes kSplitSlots workgroup slots (two per CU of
// a 256-CU device), which bounds the chunks by 4 * kSplitSlots whatever the
// device; a forced size s bounds them by rows * ceil(nb / s).
constexpr int kSplitSlots = 512;

int chunk_cap(int batch, int heads, int nb, uint32_t flags) {
  if (flags & 1u) return 0;  // one workgroup per row: nothing is split
  const int forced = (int)((flags >> 8) & 0xFFFFu);
  if (forced == 0) return 4 * kSplitSlots;
  const int64_t cap = (int64_t)batch * heads * nb * ((nb + forced - 1) / forced);
  return (int)std::min<int64_t>(cap, (int64_t)1 << 28);
}

// Query-block pairs per head under these flags: none for the naive grid,
// under FVA_SCHED_UNPAIRED and in the allocation-free call.
int pairs_of(const Geometry& g, uint32_t flags, bool lean) {
  return (lean || (flags & 5u)) ? 0 : pairs_per_head(g);
}

// lean: the layout of the allocation-free call -- no room for rebuilt counts
// and kept lists (the caller passes them), no chunk items (no row is split,
// so no partial results are kept) and no query-block pairs.
AttnWorkspace carve(void* base, int batch, int heads, const Geometry& g, uint32_t flags, bool lean = false) {
  const int nb = g.nb;
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t rows = (size_t)batch * heads * nb;
  const size_t nh = (size_t)batch * heads;
  char* p = reinterpret_cast<char*>(base);
  AttnWorkspace w;
  w.cap = lean ? 0 : chunk_cap(batch, heads, nb, flags);
  const size_t cap = (size_t)w.cap;
  size_t off = 0;
  w.counts = lean ? nullptr : reinterpret_cast<int32_t*>(p + off);
  off += lean ? 0 : al(rows * 4);
  w.kv = lean ? nullptr : reinterpret_cast<int32_t*>(p + off);
  off += lean ? 0 : al(rows * nb * 4);
  w.items = reinterpret_cast<int32_t*>(p + off);
  off += al((rows + cap) * 4);
  w.qbase = reinterpret_cast<int32_t*>(p + off);
  off += al((kQueues + 1) * 4);
  w.qctr = reinterpret_cast<int32_t*>(p + off);
  off += al(kQueues * 4);
  w.hscratch = reinterpret_cast<int32_t*>(p + off);
  off += al(nh * (2 + 2 * kQueues + 1) * 4);
  w.rscratch = reinterpret_cast<int32_t*>(p + off);
  off += al(2 * (rows + 1) * 4);
  w.n_split = reinterpret_cast<int32_t*>(p + off);
  off += al(4);
  w.chunks = reinterpret_cast<int4*>(p + off);
  off += al(cap * sizeof(int4));
  w.splits = reinterpret_cast<int4*>(p + off);
  off += al(cap * sizeof(int4));
  w.partials = reinterpret_cast<float*>(p + off);
  off += al(cap * kPartialFloats * sizeof(float));
  w.bmap = reinterpret_cast<BlockMap*>(p + off);
  off += al((size_t)nb * sizeof(BlockMap));
  w.pairs_head = pairs_of(g, flags, lean);
  const size_t pairs = nh * (size_t)w.pairs_head;
  w.plist = w.pcount = w.pfirst = w.psplit = nullptr;
  if (pairs > 0) {
    w.plist = reinterpret_cast<int32_t*>(p + off);
    off += al(pairs * nb * 4);
    w.pcount = reinterpret_cast<int32_t*>(p + off);
    off += al(pairs * 4);
    w.pfirst = reinterpret_cast<int32_t*>(p + off);
    off += al((size_t)w.pairs_head * 4);
    w.psplit = reinterpret_cast<int32_t*>(p + off);
    off += al(4);
  }
  w.bytes = off;
  return w;
}
}  // namespace

size_t attn_workspace_bytes(int batch, int heads, const Geometry& g, uint32_t flags) {
  return carve(nullptr, batch, heads, g, flags).bytes;
}

// ---- Allocation-free attention ---------------------------------------------
// The plan, queue and block-table scratch of fva_attn_noalloc lives in this
// file-scope device array (each device holds its own copy for the life of
// the process). Its device address is taken once per device with that device
// current and kept; host code passes only that address to kernels, never
// the array's name, which is a host-side stand-in.
constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

size_t attn_noalloc_bytes(int batch, int heads, const Geometry& g) {
  return carve(nullptr, batch, heads, g, 0u, true).bytes;
}

size_t attn_noalloc_capacity() { return kNoAllocScratchBytes; }

namespace {
hipError_t scratch_address(void** out) {
  static void* addr[64] = {};
  static std::mutex lock;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> guard(lock);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}
}  // namespace

int64_t attn_trace_words(int batch, int heads, int nb) {
  return 4 * ((int64_t)batch * heads * nb + 4 * kSplitSlots);
}

hipError_t launch_attn(const AttnArgs& a) {
  (void)hipGetLastError();  // drop an error left by an unrelated earlier HIP call
  const Geometry g = make_geometry(a.T, a.H, a.W, a.bt, a.bh, a.bw);
  const int n_items = a.batch * a.heads * g.nb;
  if (n_items == 0) return hipSuccess;
  const AttnWorkspace ws = carve(a.workspace, a.batch, a.heads, g, a.flags, a.lean);
  int32_t* ws_counts = ws.counts;
  int32_t* ws_kv = ws.kv;
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
  P.V8 = a.V8;
  P.vexp = a.vexp;
  const bool f8 = a.V8 != nullptr;
  P.O = reinterpret_cast<uint16_t*>(a.O);
  P.heads = a.heads;
  P.sb = a.stride_b;
  P.sh = a.stride_h;
  P.sn = a.stride_n;
  P.g = g;
  P.counts = counts;
  P.kv_idx = kv_idx;
  P.bmap = ws.bmap;
  P.chunks = ws.chunks;
  P.partials = ws.partials;
  P.n_rows = n_items;
  P.trace_chunks = 4 * kSplitSlots;
  P.c2 = a.scale * 1.4426950408889634f;
  P.trace = (a.flags & 2u) ? a.trace : nullptr;
  P.plist = ws.plist;
  P.pcount = ws.pcount;
  P.psplit = ws.psplit;
  P.pairs_head = ws.pairs_head;

  hipLaunchKernelGGL(block_table_kernel, dim3(1), dim3(1024), 0, a.stream, g, ws.bmap, ws.pfirst);
  e = hipGetLastError();
  if (e != hipSuccess) return e;

  if (a.flags & 1u) {
    if (f8)
      hipLaunchKernelGGL(attn_naive_kernel<true>, dim3(n_items), dim3(kAttnThreads), 0, a.stream, P);
    else
      hipLaunchKernelGGL(attn_naive_kernel<false>, dim3(n_items), dim3(kAttnThreads), 0, a.stream, P);
    return hipGetLastError();
  }
  const int forced = (int)((a.flags >> 8) & 0xFFFFu);
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(1024), 0, a.stream, counts, a.batch * a.heads, g, kSplitSlots, forced,
                     ws.cap, ws.items, ws.qbase, ws.qctr, ws.hscratch, ws.rscratch, ws.chunks, ws.splits, ws.n_split,
                     ws.bmap, ws.plist ? 1 : 0, ws.psplit);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (ws.plist) {
    const int n_pairs = a.batch * a.heads * ws.pairs_head;
    const int pgrid = std::max(1, std::min((n_pairs + 3) / 4, 4 * info.cus));
    hipLaunchKernelGGL(pair_list_kernel, dim3(pgrid), dim3(256), 0, a.stream, counts, kv_idx, a.batch * a.heads,
                       g.nb, ws.bmap, ws.pairs_head, ws.pfirst, ws.psplit, ws.plist, ws.pcount);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  int grid = info.cus * (f8 ? info.per_cu8 : info.per_cu);
  if ((int64_t)grid > (int64_t)n_items + ws.cap) grid = n_items + ws.cap;
  if (f8)
    hipLaunchKernelGGL(attn_persistent_kernel<true>, dim3(grid), dim3(kAttnThreads), 0, a.stream, P, ws.items,
                       ws.qbase, ws.qctr);
  else
    hipLaunchKernelGGL(attn_persistent_kernel<false>, dim3(grid), dim3(kAttnThreads), 0, a.stream, P, ws.items,
                       ws.qbase, ws.qctr);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // Split rows (if any) are merged; the workgroups beyond their number exit.
  if (g.nb > (forced > 0 ? forced : kMinChunk)) {
    const int cgrid = std::max(1, std::min(ws.cap / 2, 2 * info.cus));
    hipLaunchKernelGGL(combine_kernel, dim3(cgrid), dim3(256), 0, a.stream, P, ws.splits, ws.n_split);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_attn_noalloc(const AttnArgs& a) {
  AttnArgs b = a;
  hipError_t e = scratch_address(&b.workspace);
  if (e != hipSuccess) return e;
  b.lean = true;
  return launch_attn(b);
}

}  // namespace fva
