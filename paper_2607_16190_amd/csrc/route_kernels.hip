// Routing frontend on gfx950: block pooling and Top-p / Top-k selection.
//
// pool_kernel   -- qbar_i, kbar_i = fp64 means of Q, K over the real tokens
//                  of block i (pooled block similarities, §3.1). One workgroup
//                  per (b, h) and 8 consecutive blocks streams their rows of
//                  Q and K once (sixteen lanes per 256-byte token row) and
//                  writes the means as whole lines in MFMA operand order.
// score_kernel  -- for 16 query blocks of one (b, h): fp64 products of the
//                  means against every key block on the fp64 matrix unit,
//                  written as score rows.
// select_kernel -- per score row (one wavefront each): softmax, Top-p cut
//                  with the Top-k floor (§2.1), then the mask row, the count
//                  and the ascending kept-block list.
// sasa_budget_kernel, augment_kernel -- the slack-aware augmentation
//                  (§3.3, Eq. 7-10, read over a head -> rank map): per-rank
//                  budgets, then extra blocks appended in the same order.
//
// The Top-p cut never sorts the row. The probabilities are turned into
// fixed-point masses F_j = round(P_j * 2^52), so every partial sum is exact
// and order-free; a bucketed radix select over the scores (64 buckets per
// level, ordered from the highest score) finds the bucket in which the
// running mass first reaches T = ceil(p * 2^52), then recurses into that
// bucket until at most 64 candidates remain, whose order is then resolved
// exactly by (score desc, block id asc). P_j carries the relative error of the fp32
// exp2 (below 2^-21, so every running sum is within 1e-6 of its exact value):
// the result equals the fp64 sequential-sum definition except where a running
// sum lies within about 1e-6 of p.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fva_common.h"
#include "fva_geometry.h"
#include "fva_internal.h"

namespace fva {

namespace {

constexpr int kPoolThreads = 512;  // one wavefront per block, 8 blocks
constexpr int kSelRows = 16;         // query blocks per select workgroup
constexpr double kMassScale = 4503599627370496.0;  // 2^52

// Pooled means are stored in the operand order of the fp64 16x16x4 MFMA of
// select_kernel: per head, tiles of 16 blocks; within tile T, load step u
// (0..15) holds 64 lanes x 2 doubles, lane 16g + m carrying dims 32g + 2u and
// 32g + 2u + 1 of block 16T + m. Every operand load of a tile is one
// contiguous kilobyte, and the 8 blocks of a pool workgroup fill whole
// 128-byte lines. Blocks are padded to a multiple of 16 (the padding means
// are zero and never read as real blocks).
__host__ __device__ constexpr int padded_blocks(int nb) { return (nb + 15) & ~15; }
constexpr int kPoolBlocks = 8;  // blocks per pool workgroup (half an operand tile)

// One workgroup pools blocks 8G .. 8G + 7 of one (b, h), one wavefront per
// block: lane (slot = lane / 16, chunk c = lane % 16) sums dims 8c .. 8c+7 of
// Q and K over rows slot, slot + 4, ... in fp64 (each wave load is four whole
// 256-byte token rows), the four slots are summed across lanes, and the
// means are staged in operand order; the group's 16 KB of Q and K means are
// then written as whole lines.
// x[l] + x[l^16] + x[l^32] + x[l^48] in every lane, with the lane-swap
// instructions (both partners add the same two operands).
__device__ __forceinline__ double sum_rows4(double v) {
  uint64_t b = (uint64_t)__double_as_longlong(v);
  auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)b, (uint32_t)b, false, false);
  auto hi = __builtin_amdgcn_permlane16_swap((uint32_t)(b >> 32), (uint32_t)(b >> 32), false, false);
  v = __longlong_as_double((long long)join64(lo[0], hi[0])) + __longlong_as_double((long long)join64(lo[1], hi[1]));
  b = (uint64_t)__double_as_longlong(v);
  lo = __builtin_amdgcn_permlane32_swap((uint32_t)b, (uint32_t)b, false, false);
  hi = __builtin_amdgcn_permlane32_swap((uint32_t)(b >> 32), (uint32_t)(b >> 32), false, false);
  return __longlong_as_double((long long)join64(lo[0], hi[0])) + __longlong_as_double((long long)join64(lo[1], hi[1]));
}

constexpr int kPoolRowsPerStep = 16;  // token rows each lane loads per step
static_assert(kPoolThreads == 64 * kPoolBlocks, "one wavefront per pooled block");
__global__ __launch_bounds__(kPoolThreads) void pool_kernel(const uint16_t* __restrict__ Q,
                                                           const uint16_t* __restrict__ K, int heads,
                                                           int64_t sb, int64_t sh, int64_t sn, Geometry g,
                                                           double* __restrict__ qbar,
                                                           double* __restrict__ kbar) {
  __shared__ double stage[2][16 * 4 * kPoolBlocks * 2];  // [tensor][u][g][block][pair]
  const int wave = threadIdx.x >> 6;  // block i0 + wave
  const int lane = threadIdx.x & 63;
  const int i0 = blockIdx.x * kPoolBlocks;
  const int i = i0 + wave;
  const int bh = blockIdx.y;
  const int c = lane & 15;     // 16-byte chunk: dims 8c .. 8c+7
  const int slot = lane >> 4;  // rows slot + 4j
  double aq[8], ak[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) { aq[e] = 0.0; ak[e] = 0.0; }
  double nreal = 1.0;
  if (i < g.nb) {
    const int b = bh / heads;
    const int h = bh - b * heads;
    const int64_t base = (int64_t)b * sb + (int64_t)h * sh + c * 8;
    const BlockBox box = block_box(g, i);
    nreal = (double)box.n;
    const int jend = (box.n + 4 * kPoolRowsPerStep - 1) / (4 * kPoolRowsPerStep) * kPoolRowsPerStep;
    // For full 8x8 planes, row r = slot + 4j sits at plane j / 16, line
    // (j / 2) % 8, column slot + 4 (j % 2); in a one-line block it is token
    // x0 + r: no divisions either way.
    const bool fast = box.ey == 8 && box.ex == 8;
    const bool line = box.n == box.ex;  // consecutive tokens: row r is token x0 + r
    const int HW = g.H * g.W;
    const int tb = (box.t0 * g.H + box.y0) * g.W + box.x0 + slot;
    for (int j0 = 0; j0 < jend; j0 += kPoolRowsPerStep) {
      uint4 vq[kPoolRowsPerStep], vk[kPoolRowsPerStep];
#pragma unroll
      for (int jj = 0; jj < kPoolRowsPerStep; ++jj) {
        const int j = j0 + jj;
        const int r = slot + 4 * j;
        if (r < box.n) {
          const int tok = fast ? tb + (j >> 4) * HW + ((j >> 1) & 7) * g.W + 4 * (j & 1)
                          : line ? tb + 4 * j : box_token(g, box, r);
          const int64_t off = base + (int64_t)tok * sn;
          // streaming loads: every byte of Q and K is read once here, and
          // the caches are left to the score rows and to the attention's K/V
          typedef unsigned int u32x4_nt __attribute__((ext_vector_type(4)));
          const u32x4_nt lq = __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(Q + off));
          const u32x4_nt lk = __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(K + off));
          vq[jj] = make_uint4(lq.x, lq.y, lq.z, lq.w);
          vk[jj] = make_uint4(lk.x, lk.y, lk.z, lk.w);
        } else {
          vq[jj] = make_uint4(0, 0, 0, 0);
          vk[jj] = make_uint4(0, 0, 0, 0);
        }
      }
#pragma unroll
      for (int jj = 0; jj < kPoolRowsPerStep; ++jj) {
        const uint32_t wq[4] = {vq[jj].x, vq[jj].y, vq[jj].z, vq[jj].w};
        const uint32_t wk[4] = {vk[jj].x, vk[jj].y, vk[jj].z, vk[jj].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          aq[2 * e] += (double)bf16_lo(wq[e]);
          aq[2 * e + 1] += (double)bf16_hi(wq[e]);
          ak[2 * e] += (double)bf16_lo(wk[e]);
          ak[2 * e + 1] += (double)bf16_hi(wk[e]);
        }
      }
    }
  }
  // Sum the four slots: lanes c, c + 16, c + 32, c + 48.
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    aq[e] = sum_rows4(aq[e]);
    ak[e] = sum_rows4(ak[e]);
  }
  // Slot 0 stores the Q means, slot 1 the K means (zero for padding blocks):
  // dims 8c + 2v, 8c + 2v + 1 are pair (u, g) = (4 (c % 4) + v, c / 4).
  if (slot < 2) {
    double* st = stage[slot];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const double x0 = slot ? ak[2 * v] : aq[2 * v];
      const double x1 = slot ? ak[2 * v + 1] : aq[2 * v + 1];
      const int u = 4 * (c & 3) + v;
      double2 m2;
      m2.x = i < g.nb ? x0 / nreal : 0.0;
      m2.y = i < g.nb ? x1 / nreal : 0.0;
      *reinterpret_cast<double2*>(&st[((u * 4 + (c >> 2)) * kPoolBlocks + wave) * 2]) = m2;
    }
  }
  __syncthreads();
  // 2 x 512 chunks of 16 bytes: chunk q of a tensor is (u, g, m) = (q / 32,
  // (q / 8) % 4, q % 8); eight consecutive threads write one 128-byte line.
  const int tile = i0 >> 4;
  const int hm = (i0 >> 3) & 1;  // which 8 blocks of the 16-block tile
  const int64_t head_off = (int64_t)bh * padded_blocks(g.nb) * kHeadDim;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int q = threadIdx.x + kPoolThreads * k;  // 0 .. 1023 over both tensors
    const int t = q >> 9;
    const int qq = q & 511;
    const int u = qq >> 5, gg = (qq >> 3) & 3, m = qq & 7;
    const double2 v = *reinterpret_cast<const double2*>(&stage[t][((u * 4 + gg) * kPoolBlocks + m) * 2]);
    double* out = (t ? kbar : qbar) + head_off + ((int64_t)(tile * 16 + u) * 64 + gg * 16 + hm * 8 + m) * 2;
    *reinterpret_cast<double2*>(out) = v;
  }
}

// The score rows hold the raw products q_i . k_j; the 1/sqrt(128) score
// scale enters only here (the order of a row does not depend on it), folded
// with log2(e) into one factor.
constexpr double kLog2eOverSqrtD = 0.12751743082459868;  // log2(e) / sqrt(128)

// Unnormalised probability exp((s - smax) / sqrt(128)) of a block (s <= smax,
// raw products), evaluated with the hardware exp2 in fp32: relative error
// below 2^-21, far inside what the Top-p decision needs (the scores
// themselves, which decide the order, stay fp64). Masses below 2^-126 flush
// to zero; they are below the 2^-52 quantum of the fixed-point sums anyway.
__device__ __forceinline__ double block_exp(double s, double smax) {
  return (double)__builtin_amdgcn_exp2f((float)((s - smax) * kLog2eOverSqrtD));
}

// Nearest integer (ties to even) of x in [0, 2^52]: x + 2^52 rounds to an
// integer, and its bit pattern exceeds that of 2^52 by exactly that integer
// (also for x = 2^52, where the exponent steps up by one).
__device__ __forceinline__ uint64_t round_mass(double x) {
  return (uint64_t)__double_as_longlong(__dadd_rn(x, kMassScale)) - (uint64_t)__double_as_longlong(kMassScale);
}

// Fixed-point mass of one block: round(block_exp(s, smax) * (2^52 / Z)).
// Z >= 1 (it holds the maximum's exp(0) = 1), so the product is at most
// 2^52. Every caller evaluates exactly this expression, so a block's mass is
// the same wherever it is recomputed.
__device__ __forceinline__ uint64_t block_mass(double s, double smax, double zs) {
  return round_mass(__dmul_rn(block_exp(s, smax), zs));
}

// A bucket of the radix select holds (count << 53) + summed weight in one
// 64-bit word: weights of a row sum to at most 2^52 + nb / 2 < 2^53, and
// counts to at most 1024, so one atomic add and one scan carry both.
constexpr uint64_t kOneCount = 1ull << 53;
constexpr uint64_t kWeightBits = kOneCount - 1;

// Largest candidate set the exact ranking of select_cut takes without one
// more bucket level first.
constexpr int kRankMax = 8;

struct WaveScratch {
  uint64_t hist[64];  // packed bucket words
  double cs[64];      // candidates: score, weight, block id
  uint64_t cw[64];
  int cj[64];
  uint64_t kept[16];  // kept-block bits of the row, 64 blocks per word
};

struct Cut {
  double s;
  int j;
  int rank;  // 1-based position of the cut block in (score desc, id asc) order
};

// Finds the block q at which the running weight (fixed-point mass, or 1 per
// block when by_mass is false) first reaches thr, walking blocks in
// (score desc, id asc) order. Requires thr >= 1 and total weight >= thr.
// Each level buckets the candidates by score into 64 buckets (bucket 0 for
// the highest scores), scans the bucket words and keeps only the bucket in
// which the running weight crosses thr; once at most 64 candidates remain,
// every candidate sums the weights of those that precede it.
template <int KPL>
__device__ Cut select_cut(const double (&s)[KPL], const uint64_t (&F)[KPL], uint32_t valid, int nvalid, double smin,
                          double smax, double zs, bool by_mass, uint64_t thr, WaveScratch& ws, int lane) {
  uint32_t cand = valid;
  int ncand = nvalid;
  uint64_t W0 = 0;  // weight of the blocks ahead of every candidate
  int C0 = 0;       // their number
  double lo = smin, hi = smax;
  for (int level = 0; level < 2 * kMaxBlocks; ++level) {  // each level drops >= 1 candidate
    if (ncand <= 64 || !(hi > lo)) {
      // Gather the candidates in ascending block id order.
      int base = 0;
#pragma unroll
      for (int k = 0; k < KPL; ++k) {
        const bool is = (cand >> k) & 1u;
        const uint64_t m = __ballot(is);
        const int pos = base + lanes_below(m);
        if (is && pos < 64) {
          ws.cs[pos] = s[k];
          ws.cj[pos] = lane + 64 * k;
          ws.cw[pos] = by_mass ? F[k] : 1ull;
        }
        base += __popcll(m);
      }
      wave_sync();
      if (ncand > 64) {
        // Every candidate has the same score: they follow in id order, each
        // with the same weight, so the cut is the t-th smallest id.
        const uint64_t w = by_mass ? block_mass(hi, smax, zs) : 1ull;
        const uint64_t need = thr - W0;
        uint64_t t = (w == 0) ? (uint64_t)ncand : (need + w - 1) / w;
        if (t > (uint64_t)ncand) t = (uint64_t)ncand;
        if (t < 1) t = 1;
        int seen = 0;
        int cut_j = -1;
#pragma unroll
        for (int k = 0; k < KPL; ++k) {
          const bool is = (cand >> k) & 1u;
          const uint64_t m = __ballot(is);
          const int cntk = __popcll(m);
          if (cut_j < 0 && seen + cntk >= (int)t) {
            const int want = (int)t - seen;  // 1-based within this k
            const uint64_t at = __ballot(is && lanes_below(m) + 1 == want);
            cut_j = 64 * k + __ffsll((unsigned long long)at) - 1;
          }
          seen += cntk;
        }
        Cut c;
        c.j = cut_j;
        c.s = hi;
        c.rank = C0 + (int)t;
        return c;
      }
      // More than kRankMax candidates of distinct scores: one more bucket
      // level over them, one per lane (the rule of the levels below), so that
      // the exact ranking that follows runs over the few of the crossing
      // bucket. Compaction in lane order keeps ascending block ids.
      if (ncand > kRankMax) {
        const bool has0 = lane < ncand;
        const double s0 = has0 ? ws.cs[lane] : 0.0;
        const int j0 = has0 ? ws.cj[lane] : 0;
        const uint64_t w0 = has0 ? ws.cw[lane] : 0ull;
        const double lo0 = wave_min(has0 ? s0 : 1.0e308);
        const double hi0 = wave_max(has0 ? s0 : -1.0e308);
        if (hi0 > lo0) {
          ws.hist[lane] = 0ull;
          wave_sync();
          int b = (int)__dmul_rn(hi0 - s0, 64.0 / (hi0 - lo0));
          b = b < 0 ? 0 : (b > 63 ? 63 : b);
          atomicAdd((unsigned long long*)&ws.hist[has0 ? b : lane],
                    (unsigned long long)(has0 ? kOneCount + w0 : 0ull));
          wave_sync();
          const uint64_t hv = ws.hist[lane];
          const uint64_t inc = wave_incl_scan_u64(hv, lane);
          const uint64_t hit = __ballot(W0 + (inc & kWeightBits) >= thr);
          const int bstar = hit ? (__ffsll((unsigned long long)hit) - 1) : 63;
          const uint64_t ahead = lane_u64(inc - hv, bstar);
          W0 += ahead & kWeightBits;
          C0 += (int)(ahead >> 53);
          const bool keep = has0 && b == bstar;
          const uint64_t km = __ballot(keep);
          ncand = __popcll(km);
          if (keep) {
            const int pos = lanes_below(km);
            ws.cs[pos] = s0;
            ws.cj[pos] = j0;
            ws.cw[pos] = w0;
          }
          wave_sync();
        }
      }
      // At most kRankMax candidates (or several of one score), one per lane:
      // each sums the weights of the candidates ahead of it (read as LDS
      // broadcasts), so the crossing is the one candidate with before < thr
      // <= before + own weight.
      const bool has = lane < ncand;
      const double sl = has ? ws.cs[lane] : 0.0;
      const int jl = has ? ws.cj[lane] : 0;
      const uint64_t wl = has ? ws.cw[lane] : 0ull;
      uint64_t ahead = 0;
      int rank = 0;
      // Eight candidates per step, read unconditionally (entries past ncand
      // are masked, the arrays hold 64) and combined without branches, so
      // the step's LDS reads are in flight together.
      for (int m0 = 0; m0 < ncand; m0 += 8) {
        double sm[8];
        int jm[8];
        uint64_t wm[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          sm[u] = ws.cs[m0 + u];
          jm[u] = ws.cj[m0 + u];
          wm[u] = ws.cw[m0 + u];
        }
        // keeps the weight reads unconditional (issued with the others)
        asm volatile("" : "+v"(wm[0]), "+v"(wm[1]), "+v"(wm[2]), "+v"(wm[3]), "+v"(wm[4]), "+v"(wm[5]), "+v"(wm[6]),
                     "+v"(wm[7]));
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const bool prec = (m0 + u < ncand) & ((sm[u] > sl) | ((sm[u] == sl) & (jm[u] < jl)));
          ahead += prec ? wm[u] : 0ull;
          rank += (int)prec;
        }
      }
      const uint64_t before = W0 + ahead;
      uint64_t hit = __ballot(has && before < thr && before + wl >= thr);
      if (!hit) hit = __ballot(has && rank == ncand - 1);  // not reached: thr is within the total
      const int pos = __ffsll((unsigned long long)hit) - 1;
      Cut c;
      c.j = __builtin_amdgcn_readlane(jl, pos);
      c.s = __longlong_as_double((long long)lane_u64((uint64_t)__double_as_longlong(sl), pos));
      c.rank = C0 + __builtin_amdgcn_readlane(rank, pos) + 1;
      wave_sync();
      return c;
    }
    // Bucket floor((hi - s) * 64 / (hi - lo)) is non-decreasing as s falls;
    // any positive scale keeps that order, so it need not be exact.
    ws.hist[lane] = 0ull;
    wave_sync();
    const double scale = 64.0 / (hi - lo);
    int bk[KPL];
#pragma unroll
    for (int k = 0; k < KPL; ++k) {
      const bool is = (cand >> k) & 1u;
      int b = (int)__dmul_rn(hi - s[k], scale);
      b = b < 0 ? 0 : (b > 63 ? 63 : b);
      bk[k] = b;
      // Lanes without a candidate add 0 to their own word: no branch and no
      // address conflict.
      atomicAdd((unsigned long long*)&ws.hist[is ? b : lane],
                (unsigned long long)(is ? kOneCount + (by_mass ? F[k] : 1ull) : 0ull));
    }
    wave_sync();
    const uint64_t hv = ws.hist[lane];
    const uint64_t inc = wave_incl_scan_u64(hv, lane);
    const uint64_t hit = __ballot(W0 + (inc & kWeightBits) >= thr);
    const int bstar = hit ? (__ffsll((unsigned long long)hit) - 1) : 63;
    const uint64_t ahead = lane_u64(inc - hv, bstar);
    W0 += ahead & kWeightBits;
    C0 += (int)(ahead >> 53);
    ncand = (int)(lane_u64(hv, bstar) >> 53);
    wave_sync();
    double nlo = 1.0e308, nhi = -1.0e308;
#pragma unroll
    for (int k = 0; k < KPL; ++k) {
      const bool keep = ((cand >> k) & 1u) && bk[k] == bstar;
      cand = keep ? cand : (cand & ~(1u << k));
      nlo = keep ? fmin(nlo, s[k]) : nlo;
      nhi = keep ? fmax(nhi, s[k]) : nhi;
    }
    if (ncand > 64) {
      lo = wave_min(nlo);
      hi = wave_max(nhi);
    }
  }
  // Not reached for finite scores; keep every block as a safe fallback.
  Cut c;
  c.j = -1;
  c.s = -1.0e308;
  c.rank = 0;
  return c;
}

template <int KPL>
__device__ __forceinline__ void emit_row(const double (&s)[KPL], int nb, int m, const Cut& cut,
                                         uint8_t* __restrict__ mrow, int32_t* __restrict__ count_out,
                                         int32_t* __restrict__ kvrow, WaveScratch& ws, int lane);

// Cut of a routed row, kept for the slack-aware augmentation: the score and
// id of its last kept block.
struct RowCut {
  double s;
  int j;
  int pad;
};

template <int KPL>
__device__ __forceinline__ void select_row(const double* __restrict__ srow, int nb, double p, int k_min,
                                           uint8_t* __restrict__ mrow, int32_t* __restrict__ count_out,
                                           int32_t* __restrict__ kvrow, WaveScratch& ws, int lane,
                                           int m_force = -1, RowCut* cut_out = nullptr) {
  double s[KPL];
  uint64_t F[KPL];
  uint32_t valid = 0;
  double vmax = -1.0e308, vmin = 1.0e308;
  // All KPL loads of a lane are issued before any is used (lanes past the
  // row re-read its last score, so no load is conditional), so the row waits
  // for one memory latency rather than KPL dependent ones. Each score row is
  // read once here.
#pragma unroll
  for (int k = 0; k < KPL; ++k) s[k] = __builtin_nontemporal_load(srow + min(lane + 64 * k, nb - 1));
#pragma unroll
  for (int k = 0; k < KPL; ++k) {
    const bool in = lane + 64 * k < nb;
    valid |= in ? 1u << k : 0u;
    s[k] = in ? s[k] : -1.0e308;
    vmax = fmax(vmax, s[k]);
    vmin = in ? fmin(vmin, s[k]) : vmin;
  }
  const double smax = wave_max(vmax);
  const double smin = wave_min(vmin);
  // F[k] first holds block_exp(s, smax) (as bits), then the fixed-point
  // mass; block_mass evaluates the same two roundings.
  double e = 0.0;
#pragma unroll
  for (int k = 0; k < KPL; ++k) {
    const double x = ((valid >> k) & 1u) ? block_exp(s[k], smax) : 0.0;
    F[k] = (uint64_t)__double_as_longlong(x);
    e += x;
  }
  const double Z = wave_sum(e);
  const double zs = __ddiv_rn(kMassScale, Z);
  uint64_t tot = 0;
#pragma unroll
  for (int k = 0; k < KPL; ++k) {
    F[k] = ((valid >> k) & 1u) ? round_mass(__dmul_rn(__longlong_as_double((long long)F[k]), zs)) : 0ull;
    tot += F[k];
  }
  const uint64_t total = wave_sum_u64(tot);

  const int kf = k_min < nb ? k_min : nb;
  int m_p;
  Cut cut;
  cut.j = -1;
  cut.s = 0.0;
  cut.rank = 0;
  if (m_force >= 0) {
    // a given count: the first m_force blocks of the same order
    m_p = m_force < nb ? m_force : nb;
  } else if (p >= 1.0) {
    m_p = nb;
  } else {
    const uint64_t T = (uint64_t)ceil(p * kMassScale);
    if (T == 0) {
      m_p = 0;
    } else if (total < T) {
      m_p = nb;
    } else {
      cut = select_cut<KPL>(s, F, valid, nb, smin, smax, zs, true, T, ws, lane);
      m_p = cut.rank;
    }
  }
  const int m = m_force >= 0 ? m_p : (m_p > kf ? m_p : kf);
  if (m > 0 && m < nb && (m != m_p || m_force >= 0))
    cut = select_cut<KPL>(s, F, valid, nb, smin, smax, zs, false, (uint64_t)m, ws, lane);
  if (cut_out && lane == 0) {
    // the row's last kept block in (score desc, id asc) order; none kept:
    // +inf, so that every block ranks after it
    cut_out->s = m <= 0 ? (double)INFINITY : m >= nb ? -(double)INFINITY : cut.s;
    cut_out->j = m <= 0 ? -1 : m >= nb ? nb : cut.j;
  }
  emit_row<KPL>(s, nb, m, cut, mrow, count_out, kvrow, ws, lane);
}

// Writes a row's mask, kept-block list and count: the first m blocks of
// (score desc, id asc), i.e. those ahead of or equal to the cut block.
template <int KPL>
__device__ __forceinline__ void emit_row(const double (&s)[KPL], int nb, int m, const Cut& cut,
                                         uint8_t* __restrict__ mrow, int32_t* __restrict__ count_out,
                                         int32_t* __restrict__ kvrow, WaveScratch& ws, int lane) {
  uint64_t mine = 0;  // lane k < KPL holds the kept bits of blocks 64k .. 64k+63
  int base = 0;
#pragma unroll
  for (int k = 0; k < KPL; ++k) {
    const int j = lane + 64 * k;
    bool kept;
    if (m <= 0) kept = false;
    else if (m >= nb) kept = true;
    else kept = (s[k] > cut.s) || (s[k] == cut.s && j <= cut.j);
    kept = kept && (j < nb);
    const uint64_t bal = __ballot(kept);
    mine = lane == k ? bal : mine;
    if (kvrow && kept) kvrow[base + lanes_below(bal)] = j;
    base += __popcll(bal);
  }
  if ((nb & 3) == 0 && (reinterpret_cast<uintptr_t>(mrow) & 3) == 0) {
    // 4-byte aligned row of whole words: lane L writes bytes 4w .. 4w+3,
    // w = L + 64i, expanding four kept bits into four 0/1 bytes.
    if (lane < KPL) ws.kept[lane] = mine;
    wave_sync();
    uint32_t* mw = reinterpret_cast<uint32_t*>(mrow);
    for (int w = lane; 4 * w < nb; w += 64) {
      const uint32_t nib = (uint32_t)(ws.kept[w >> 4] >> (4 * (w & 15))) & 0xFu;
      mw[w] = (nib * 0x204081u) & 0x01010101u;
    }
    wave_sync();
  } else {
#pragma unroll
    for (int k = 0; k < KPL; ++k) {
      const int j = lane + 64 * k;
      const uint64_t bal = lane_u64(mine, k);
      if (j < nb) mrow[j] = (bal >> lane) & 1u;
    }
  }
  if (lane == 0) *count_out = m;
}

typedef double f64x4 __attribute__((ext_vector_type(4)));
constexpr int kScoreThreads = 256;  // 4 waves; several workgroups per CU overlap their tile loads
constexpr int kRowWaves = 4;        // rows (one per wavefront) per select workgroup

// Workgroup n of a 1-D grid runs on XCD n % 8. Logical workgroups are dealt
// out so that each XCD takes one contiguous run of them: the query tiles of
// whole heads, whose pooled keys then stay in that XCD's L2.
__device__ __forceinline__ int xcd_contiguous(int n, int total) {
  const int q = total >> 3, r = total & 7, x = n & 7;
  return x * q + min(x, r) + (n >> 3);
}

// Raw products qbar_i . kbar_j (the score s_ij times sqrt(128)) of 16 query
// blocks against every key block with the fp64 MFMA (16x16x4): lane (row
// l%16, group g = l/16) feeds dim 32g + k of its query row and its key at
// step k, so the 32 steps sum the full 128-dim dot product. Wave w takes key
// tiles w, w+4, ... The grid is one-dimensional over (head, query tile); the
// products go to a row-major [B*H*nb, nb] fp64 buffer.
__global__ __launch_bounds__(kScoreThreads, 3) void score_kernel(const double* __restrict__ qbar,
                                                             const double* __restrict__ kbar, int nb,
                                                             double* __restrict__ scores) {
  const int ntq = (nb + kSelRows - 1) / kSelRows;
  const int L = xcd_contiguous(blockIdx.x, gridDim.x);
  const int bh = L / ntq;
  const int tq = L - bh * ntq;  // query tile
  const int i0 = tq * kSelRows;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwaves = kScoreThreads / 64;
  const int m16 = lane & 15;
  const int g = lane >> 4;

  // Operands in the order written by pool_kernel: MFMA step k = 2u + e of
  // lane (m16, g) multiplies dim 32g + 2u + e of query row m16 and key m16 of
  // the tile; each load is one contiguous kilobyte. Rows and keys of the last
  // tile past nb are padding (zero means): their scores are never stored.
  const int ntiles = (nb + 15) >> 4;
  const int64_t head_off = (int64_t)bh * padded_blocks(nb) * kHeadDim;
  double qa[32];
  {
    const double* qr = qbar + head_off + (int64_t)tq * 16 * kHeadDim + 2 * lane;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const double2 v = *reinterpret_cast<const double2*>(qr + u * 128);
      qa[2 * u] = v.x;
      qa[2 * u + 1] = v.y;
    }
  }
  const double* kb = kbar + head_off + 2 * lane;
  double* srow = scores + ((int64_t)bh * nb + i0) * nb;
  auto load_tile = [&](int t, double (&kk)[32]) {
    const double* kr = kb + (int64_t)t * 16 * kHeadDim;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const double2 v = *reinterpret_cast<const double2*>(kr + u * 128);
      kk[2 * u] = v.x;
      kk[2 * u + 1] = v.y;
    }
  };
  auto score_tile = [&](int t, const double (&kk)[32]) {
    f64x4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int k = 0; k < 32; ++k) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[k], kk[k], acc, 0, 0, 0);
    // D layout of the fp64 16x16x4 MFMA: lane holds rows g + 4e (e = 0..3)
    // of key column m16; sixteen lanes store 128 contiguous bytes of a row.
    const int key = t * 16 + m16;
    if (key < nb) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = g + 4 * e;
        if (i0 + r < nb) srow[(int64_t)r * nb + key] = acc[e];
      }
    }
  };
  // One key tile in registers at a time (104 VGPRs, so four waves per SIMD):
  // they hide each other's tile loads better than two waves that each
  // double-buffer their tiles.
  double ka[32];
  for (int t = wave; t < ntiles; t += nwaves) {
    load_tile(t, ka);
    score_tile(t, ka);
  }
}

// Top-p / Top-k selection of one score row per wavefront.
template <int KPL>
__global__ __launch_bounds__(64 * kRowWaves, KPL > 12 ? 3 : 4) void select_kernel(const double* __restrict__ scores, int nb,
                                                                   int64_t nrows, double p, int k_min,
                                                                   uint8_t* __restrict__ mask,
                                                                   int32_t* __restrict__ counts,
                                                                   int32_t* __restrict__ kv_idx,
                                                                   RowCut* __restrict__ cuts) {
  __shared__ WaveScratch wsa[kRowWaves];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t row = (int64_t)blockIdx.x * kRowWaves + wave;
  if (row >= nrows) return;
  select_row<KPL>(scores + row * nb, nb, p, k_min, mask + row * nb, counts + row, kv_idx ? kv_idx + row * nb : nullptr,
                  wsa[wave], lane, -1, cuts ? cuts + row : nullptr);
}

// Slack-aware augmentation, second pass: a row of a head with extra[h] > 0
// keeps the first min(nb, counts + extra) blocks of the same order (the
// scores are those of the first pass); other rows are left as they are. The
// first pass recorded each row's last kept block, so the blocks to add are
// the first `extra` of those ranked after it: a count selection among them
// alone, with no probabilities (the order is the scores').
template <int KPL>
__global__ __launch_bounds__(64 * kRowWaves, KPL > 12 ? 3 : 4) void augment_kernel(
    const double* __restrict__ scores, int nb, int64_t nrows, const int32_t* __restrict__ extra,
    const RowCut* __restrict__ cuts, uint8_t* __restrict__ mask, int32_t* __restrict__ counts,
    int32_t* __restrict__ kv_idx) {
  __shared__ WaveScratch wsa[kRowWaves];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t row = (int64_t)blockIdx.x * kRowWaves + wave;
  if (row >= nrows) return;
  // The head's extra count, the row's count and its cut do not depend on one
  // another: loaded together, ahead of the test that needs the first two.
  const int e = __builtin_amdgcn_readfirstlane(extra[row / nb]);
  const int c0 = __builtin_amdgcn_readfirstlane(counts[row]);
  const RowCut rc = cuts[row];
  const double s_cut = rc.s;
  const int j_cut = __builtin_amdgcn_readfirstlane(rc.j);
  asm volatile("" ::"v"(s_cut), "s"(j_cut));
  const int m0 = min(max(c0, 0), nb);
  if ((e <= 0) | (m0 >= nb)) return;
  const double* srow = scores + row * nb;
  double s[KPL];
  uint64_t F[KPL];
  uint32_t cand = 0;
  double cmax = -1.0e308, cmin = 1.0e308;
  // every load of the row in flight at once, as in select_row
#pragma unroll
  for (int k = 0; k < KPL; ++k) s[k] = srow[min(lane + 64 * k, nb - 1)];
#pragma unroll
  for (int k = 0; k < KPL; ++k) {
    const int j = lane + 64 * k;
    F[k] = 0ull;
    const bool in = j < nb;
    s[k] = in ? s[k] : -1.0e308;
    const bool c = in && (s[k] < s_cut || (s[k] == s_cut && j > j_cut));
    cand |= c ? 1u << k : 0u;
    cmax = c ? fmax(cmax, s[k]) : cmax;
    cmin = c ? fmin(cmin, s[k]) : cmin;
  }
  int ncand = 0;
#pragma unroll
  for (int k = 0; k < KPL; ++k) ncand += __popcll(__ballot((cand >> k) & 1u));
  const int add = min(e, ncand);
  const int m = m0 + add;
  Cut cut;
  cut.s = s_cut;
  cut.j = j_cut;
  cut.rank = m0;
  if (add > 0 && add < ncand) {
    cut = select_cut<KPL>(s, F, cand, ncand, wave_min(cmin), wave_max(cmax), 0.0, false, (uint64_t)add, wsa[wave],
                          lane);
  } else if (add > 0) {
    cut.s = -1.0e308;  // every candidate joins: the row keeps all its blocks
    cut.j = nb;
  }
  emit_row<KPL>(s, nb, m >= nb ? nb : m, cut, mask + row * nb, counts + row, kv_idx ? kv_idx + row * nb : nullptr,
                wsa[wave], lane);
}

// Slack-aware augmentation, budget (one workgroup): S_h = kept blocks of head
// h over its rows, S_r = sum over the heads of rank r (exact integers),
// S_max = max_r S_r; a rank whose slack D = S_max - S_r passes the trigger
// D > n2 * S_max gets floor(n1 * D / (nb * H_r)) extra blocks per row (H_r
// heads). Heads with a rank id outside [0, n_ranks) take no part.
constexpr int kMaxRanks = 1024;

__global__ __launch_bounds__(1024) void sasa_budget_kernel(const int32_t* __restrict__ counts, int n_heads, int nb,
                                                           const int32_t* __restrict__ rank_of, int n_ranks,
                                                           double n1, double n2, int32_t* __restrict__ extra_head,
                                                           int32_t* __restrict__ rank_extra) {
  __shared__ unsigned long long S_r[kMaxRanks];
  __shared__ int H_r[kMaxRanks];
  __shared__ int ex_r[kMaxRanks];
  __shared__ unsigned long long S_max;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  for (int r = threadIdx.x; r < n_ranks; r += blockDim.x) {
    S_r[r] = 0ull;
    H_r[r] = 0;
  }
  __syncthreads();
  for (int h = wave; h < n_heads; h += nwaves) {
    // nb <= kMaxBlocks: a lane's counts of the head, all loads in flight at once
    const int32_t* crow = counts + (int64_t)h * nb;
    int c[kMaxBlocks / 64];
#pragma unroll
    for (int k = 0; k < kMaxBlocks / 64; ++k) c[k] = crow[min(lane + 64 * k, nb - 1)];
    unsigned long long sum = 0ull;
#pragma unroll
    for (int k = 0; k < kMaxBlocks / 64; ++k) {
      const int ck = c[k] < 0 ? 0 : (c[k] > nb ? nb : c[k]);
      sum += lane + 64 * k < nb ? (unsigned long long)ck : 0ull;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    const int r = rank_of[h];
    if (lane == 0 && r >= 0 && r < n_ranks) {
      atomicAdd(&S_r[r], sum);
      atomicAdd(&H_r[r], 1);
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long mx = 0ull;
    for (int r = 0; r < n_ranks; ++r) mx = S_r[r] > mx ? S_r[r] : mx;
    S_max = mx;
  }
  __syncthreads();
  for (int r = threadIdx.x; r < n_ranks; r += blockDim.x) {
    const unsigned long long D = S_max - S_r[r];
    int e = 0;
    if (H_r[r] > 0 && (double)D > n2 * (double)S_max) e = (int)floor((n1 * (double)D) / (double)(nb * H_r[r]));
    ex_r[r] = e;
    if (rank_extra) rank_extra[r] = e;
  }
  __syncthreads();
  for (int h = threadIdx.x; h < n_heads; h += blockDim.x) {
    const int r = rank_of[h];
    extra_head[h] = (r >= 0 && r < n_ranks) ? ex_r[r] : 0;
  }
}

template <int KPL>
hipError_t launch_select(const RouteArgs& a, int nb, const double* scores) {
  const int64_t nrows = (int64_t)a.batch * a.heads * nb;
  const dim3 grid((unsigned)((nrows + kRowWaves - 1) / kRowWaves));
  hipLaunchKernelGGL(select_kernel<KPL>, grid, dim3(64 * kRowWaves), 0, a.stream, scores, nb, nrows, a.p, a.k_min,
                     a.mask, a.counts, a.kv_idx, a.rank_of ? reinterpret_cast<RowCut*>(a.row_cuts) : nullptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !a.rank_of) return e;
  hipLaunchKernelGGL(sasa_budget_kernel, dim3(1), dim3(1024), 0, a.stream, a.counts, a.batch * a.heads, nb, a.rank_of,
                     a.n_ranks, a.n1, a.n2, a.extra_head, a.rank_extra);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(augment_kernel<KPL>, grid, dim3(64 * kRowWaves), 0, a.stream, scores, nb, nrows, a.extra_head,
                     reinterpret_cast<const RowCut*>(a.row_cuts), a.mask, a.counts, a.kv_idx);
  return hipGetLastError();
}

// Workspace: pooled Q means, pooled K means (operand order, blocks padded to
// 16), then the fp64 score rows; each part 256-byte aligned.
struct RouteWorkspace {
  size_t means;   // bytes of one means array
  size_t scores;  // bytes of the score rows
};
RouteWorkspace route_workspace_parts(int batch, int heads, int nb) {
  RouteWorkspace w;
  w.means = ((size_t)batch * heads * padded_blocks(nb) * kHeadDim * sizeof(double) + 255) & ~(size_t)255;
  w.scores = ((size_t)batch * heads * nb * nb * sizeof(double) + 255) & ~(size_t)255;
  return w;
}

}  // namespace

size_t route_workspace_bytes(int batch, int heads, int nb) {
  const RouteWorkspace w = route_workspace_parts(batch, heads, nb);
  return 2 * w.means + w.scores;
}

size_t route_sasa_workspace_bytes(int batch, int heads, int nb) {
  return route_workspace_bytes(batch, heads, nb) + (((size_t)batch * heads * 4 + 255) & ~(size_t)255) +
         (((size_t)batch * heads * nb * sizeof(RowCut) + 255) & ~(size_t)255);
}

hipError_t launch_route(const RouteArgs& a) {
  (void)hipGetLastError();  // drop an error left by an unrelated earlier HIP call
  const Geometry g = make_geometry(a.T, a.H, a.W, a.bt, a.bh, a.bw);
  const int bhs = a.batch * a.heads;
  if (bhs == 0) return hipSuccess;
  const RouteWorkspace w = route_workspace_parts(a.batch, a.heads, g.nb);
  char* base = reinterpret_cast<char*>(a.workspace);
  double* qbar = reinterpret_cast<double*>(base);
  double* kbar = reinterpret_cast<double*>(base + w.means);
  double* scores = reinterpret_cast<double*>(base + 2 * w.means);
  RouteArgs args = a;
  if (a.rank_of) {
    args.extra_head = reinterpret_cast<int32_t*>(base + 2 * w.means + w.scores);
    args.row_cuts = base + 2 * w.means + w.scores + (((size_t)bhs * 4 + 255) & ~(size_t)255);
  }
  hipLaunchKernelGGL(pool_kernel, dim3(padded_blocks(g.nb) / kPoolBlocks, bhs), dim3(kPoolThreads), 0, a.stream,
                     reinterpret_cast<const uint16_t*>(a.Q), reinterpret_cast<const uint16_t*>(a.K), a.heads,
                     a.stride_b, a.stride_h, a.stride_n, g, qbar, kbar);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(score_kernel, dim3((g.nb + kSelRows - 1) / kSelRows * bhs), dim3(kScoreThreads), 0, a.stream,
                     qbar, kbar, g.nb, scores);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int kpl = (g.nb + 63) / 64;
  if (kpl <= 2) return launch_select<2>(args, g.nb, scores);
  if (kpl <= 4) return launch_select<4>(args, g.nb, scores);
  if (kpl <= 8) return launch_select<8>(args, g.nb, scores);
  if (kpl <= 12) return launch_select<12>(args, g.nb, scores);
  return launch_select<16>(args, g.nb, scores);
}

}  // namespace fva
