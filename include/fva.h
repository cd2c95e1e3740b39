/*
 * fva.h -- C ABI of the MI355X (gfx950) Top-p block-sparse video attention
 * library (libfva.so).
 *
 * The library implements the per-step hot path of FVAttn's sparse attention
 * ("Adaptive Sparse Attention with Runtime Load Balancing for Video
 * Generation"): the routing frontend of §3.1 (video-aware 3D blocks,
 * pooled block similarities, Top-p with a Top-k floor, §2.1) and
 * block-sparse attention over the retained blocks (§2.1, §3.1), with the
 * Hilbert-curve block order of §3.1 as an alternative block organisation.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Q, K, V, O are bf16 tensors of shape [batch, heads, tokens, head_dim]
 *   with element strides (stride_b, stride_h, stride_n) and a contiguous
 *   head_dim. All four use the strides of one fva_qkv_desc.
 * - Tokens of a T x H x W latent grid are in raster order,
 *   n = (t*H + y)*W + x. Blocks are bt x bh x bw boxes anchored at the
 *   origin (a partial box only at the end of an axis); block ids are raster
 *   order over the box grid; nb = ceil(T/bt)*ceil(H/bh)*ceil(W/bw). A block
 *   holds only its real tokens (n_i <= bt*bh*bw); padding is never read.
 * - Device pointers are device memory of the current HIP device; the
 *   descriptor and tiling structs are host memory read during the call.
 * - Ownership: the caller owns every buffer. The library keeps no state
 *   between calls and allocates nothing; scratch space is the explicit
 *   workspace, whose size the *_workspace_size queries return.
 * - Asynchrony: every launching call is asynchronous on `stream` (a
 *   hipStream_t; NULL is the default stream). It reads no device data on the
 *   host and never synchronises; outputs are valid once the stream has
 *   reached the call.
 * - Errors: arguments are validated on the host before anything is
 *   launched. On a negative status nothing was launched and no output was
 *   written. FVA_ERR_HIP reports a failed kernel launch.
 * - Reentrancy: calls may overlap on different streams if their workspaces
 *   and outputs are distinct.
 * - Supported shapes: head_dim == 128, bt*bh*bw in {64, 128}, nb <= 1024,
 *   tokens * stride_n * 2 < 2^31 (one head addressed with 32-bit byte
 *   offsets), batch * heads <= 65535 for the routing calls,
 *   fva_quantize_v and fva_permute_tokens, and for the attention calls
 *   batch * heads * nb plus the chunk items (2048 with the automatic chunk
 *   size, 2^28 under FVA_SPLIT_BLOCKS, none under FVA_SCHED_NAIVE) below 2^31
 *   (32-bit work-item indices). Anything else returns FVA_ERR_UNSUPPORTED
 *   (there is no slow generic path).
 * - Utility calls (fva_num_blocks, the *_workspace_size and size queries,
 *   fva_trace_words, fva_status_string) are bookkeeping of this interface:
 *   no passage of the paper defines them.
 */
#ifndef FVA_H
#define FVA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fva_status {
  FVA_OK = 0,
  FVA_ERR_INVALID_ARG = -1, /* null pointer, p outside [0,1] or NaN, k_min < 0, bad flags */
  FVA_ERR_SHAPE = -2,       /* tokens != T*H*W, non-positive extents, bad strides */
  FVA_ERR_UNSUPPORTED = -3, /* head_dim != 128, tile volume not 64/128, nb > 1024, head > 2 GiB,
                               curve grid extent > 256, batch*heads > 65535 where noted,
                               attention work items >= 2^31 */
  FVA_ERR_WORKSPACE = -4,   /* workspace missing or smaller than the query says */
  FVA_ERR_HIP = -5,         /* a kernel launch failed */
  FVA_ERR_SCRATCH = -6      /* fva_attn_noalloc: the shape needs more than the static scratch */
} fva_status;

/* Latent grid (T x H x W) and 3D block box (bt x bh x bw). */
typedef struct fva_tiling {
  int32_t T, H, W;
  int32_t bt, bh, bw;
} fva_tiling;

/* Shape and element strides of Q, K, V and O ([batch, heads, tokens, head_dim]). */
typedef struct fva_qkv_desc {
  int32_t batch, heads, tokens, head_dim;
  int64_t stride_b, stride_h, stride_n; /* in elements; head_dim stride is 1 */
} fva_qkv_desc;

/* fva_attn flags. */
#define FVA_SCHED_PERSISTENT 0u /* persistent grid pulling (head, query-block) items, heaviest first */
#define FVA_SCHED_NAIVE 1u      /* one workgroup per item in head-major order (same kernel body) */
#define FVA_TRACE 2u            /* record per-item start/end clock and CU id into `trace` */
/* Persistent scheduler only: run every query block as an item of its own.
 * Without it, two neighbouring query blocks that both hold at most 64 real
 * tokens and are both unsplit run as one 128-row item over the union of
 * their kept lists (each block on two of the four waves, each wave skipping
 * the key blocks its block does not keep), so that every K/V tile either
 * keeps is staged once. Neighbours are x-neighbours (ix, ix + 1), ix even,
 * of one (t, y) line; among the blocks no such pair holds, y-neighbours
 * (iy, iy + 1), iy even, of one (t, x) column. Each row still sees exactly
 * its own key blocks in ascending order: the output is the same bit for
 * bit. */
#define FVA_SCHED_UNPAIRED 4u
/* Persistent scheduler only: split every row keeping more than s blocks into
 * ceil(count / s) chunk items of at most s blocks (1 <= s <= 65535). Without
 * it the chunk size is automatic: max(32, ceil(total / 1024)) with total the
 * sum over rows of (kept blocks + 1), so rows are split only when there are
 * few of them per workgroup slot. */
#define FVA_SPLIT_BLOCKS(s) (((uint32_t)(s) & 0xFFFFu) << 8)

/* Number of blocks of a tiling, or -1 if an extent is not positive. Host only. */
int32_t fva_num_blocks(const fva_tiling* tiling);

/*
 * Workspace bytes needed by fva_route for this shape: the pooled block means
 * of Q and K in fp64 with nb rounded up to a multiple of 16
 * (2 * batch*heads*ceil16(nb)*128*8 bytes) and the fp64 block scores
 * (batch*heads*nb*nb*8 bytes), each part 256-byte aligned.
 */
fva_status fva_route_workspace_size(const fva_qkv_desc* desc, const fva_tiling* tiling, size_t* bytes);

/*
 * fva_route -- routing frontend (§3.1; Top-p and the Top-k floor of §2.1).
 *
 * For every (b, h) and query block i:
 *   qbar_i, kbar_j = means of Q and K over the real tokens of each block;
 *   s_ij = qbar_i . kbar_j / sqrt(128), P_ij = softmax over all j of s_ij;
 *   key blocks ordered by decreasing s_ij (ties: lower j first), c_r the
 *   running sum of their P; m_p = min{r : c_r >= p} (nb if none reaches p,
 *   and nb when p == 1); m = max(m_p, min(k_min, nb)); the first m blocks of
 *   that order are kept.
 * Pooling and scores are fp64, so the order of the key blocks is exact. The
 * probabilities use an fp32 exp2 (relative error below 2^-21) and are summed
 * as exact fixed-point masses (2^-52 quanta), so the decision c_r >= p agrees
 * with an fp64 sequential sum except within about 1e-6 of p.
 *
 * Inputs : Q, K (bf16, desc), p in [0, 1], k_min >= 0, tiling. Q and K are
 *          taken to be finite: with NaN or infinite elements the call still
 *          writes every output in bounds and returns, but which blocks a
 *          row keeps is unspecified.
 * Outputs: block_mask uint8 [batch, heads, nb, nb] (1 = kept), fully written;
 *          counts int32 [batch, heads, nb] = m per row, fully written;
 *          kv_idx int32 [batch, heads, nb, nb] or NULL: row (b,h,i) holds the
 *          kept block ids in ascending order in its first counts[b,h,i]
 *          entries; later entries are left untouched.
 * workspace: at least fva_route_workspace_size bytes of device memory,
 *          256-byte aligned.
 * Errors : as in the conventions above; FVA_ERR_UNSUPPORTED also for
 *          batch * heads > 65535.
 */
fva_status fva_route(const void* Q, const void* K, const fva_qkv_desc* desc, double p, int32_t k_min,
                     const fva_tiling* tiling, uint8_t* block_mask, int32_t* counts, int32_t* kv_idx,
                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * Slack-aware sparse augmentation (§3.3), for the heads one GPU holds,
 * grouped into ranks by rank_of.
 *
 * After routing as fva_route does, with S_h the sum of counts over head h's
 * rows (nb * L_h of Eq. 1), S_r the sum of S_h over the heads of rank r and
 * S_max = max_r S_r: a rank whose slack D_r = S_max - S_r passes the trigger
 * D_r > n2 * S_max (the paper's threshold n2 on the slack) gets the budget
 * n1 * D_r / nb rows of work (the budget B_r = n1 * slack), spent evenly:
 * every row of its H_r heads keeps
 *   e_r = floor((n1 * D_r) / (nb * H_r))
 * more key blocks, the next ones in the routing order (score descending,
 * ties to the lower id); a row never keeps more than nb. The trigger and
 * e_r are evaluated in fp64 exactly as written, from exact integer sums, so
 * the result is deterministic; the rank loads S_r + H_r * nb * e_r never
 * exceed S_max (no new straggler, n1 <= 1).
 */
/* Workspace of fva_route_sasa: that of fva_route, plus batch*heads int32
 * (extra blocks per head) and a 16-byte record per routed row (the row's
 * last kept block after the first pass, from which the augmentation ranks
 * the blocks after it), each part 256-byte aligned. Host only. */
fva_status fva_route_sasa_workspace_size(const fva_qkv_desc* desc, const fva_tiling* tiling, size_t* bytes);

/*
 * fva_route_sasa -- fva_route followed by the augmentation above.
 * rank_of: device int32 [batch * heads], the rank of head (b, h) at index
 *          b * heads + h; heads with an id outside [0, n_ranks) take no
 *          part (no load, no extra blocks).
 * n_ranks in [1, 1024]; n1, n2 in [0, 1] (the paper uses 0.8 and 0.07).
 * Outputs as for fva_route (after augmentation); rank_extra: device int32
 *          [n_ranks] = e_r, or NULL.
 * Errors as for fva_route; FVA_ERR_INVALID_ARG for a NULL or misaligned
 * rank_of, n_ranks or n1 / n2 out of range.
 */
fva_status fva_route_sasa(const void* Q, const void* K, const fva_qkv_desc* desc, double p, int32_t k_min,
                          const fva_tiling* tiling, const int32_t* rank_of, int32_t n_ranks, double n1, double n2,
                          uint8_t* block_mask, int32_t* counts, int32_t* kv_idx, int32_t* rank_extra, void* workspace,
                          size_t workspace_bytes, void* stream);

/*
 * Workspace bytes needed by fva_attn for this shape and flags: the work
 * list and queue counters, room for counts and kv_idx (batch*heads*nb and
 * batch*heads*nb*nb int32) used when the caller passes them as NULL, one
 * 32-byte record per block, the partial results of split rows: 66,560
 * bytes per chunk for at most 2048 chunks (automatic chunk size) or
 * batch*heads*nb*ceil(nb/s) chunks under FVA_SPLIT_BLOCKS(s), none under
 * FVA_SCHED_NAIVE; and the union lists of the query-block pairs,
 * batch*heads*P*(nb + 1) int32 with P the pairs a head holds (none under
 * FVA_SCHED_NAIVE or FVA_SCHED_UNPAIRED).
 */
fva_status fva_attn_workspace_size(const fva_qkv_desc* desc, const fva_tiling* tiling, uint32_t flags,
                                   size_t* bytes);

/* Number of int64 words `trace` must hold under FVA_TRACE: 4 per (b, h, i)
 * row, then 4 for each of up to 2048 chunk items of split rows; -1 for a
 * shape the attention calls do not support. */
int64_t fva_trace_words(const fva_qkv_desc* desc, const fva_tiling* tiling);

/*
 * fva_attn -- block-sparse attention over the retained blocks (§2.1: only
 * the selected query-key block pairs are evaluated; §3.1).
 *
 * For every real query token n of block i of (b, h):
 *   O_n = sum over the real tokens k of every key block j with
 *         block_mask[b,h,i,j] = 1 of softmax_k(softmax_scale * Q_n . K_k) V_k,
 * and O_n = 0 when the row keeps no block. bf16 MFMA products, fp32
 * accumulation and softmax statistics, bf16 output.
 *
 * block_mask: uint8 [batch, heads, nb, nb], any 0/1 pattern.
 * counts, kv_idx: either both NULL (they are rebuilt from block_mask in the
 *          workspace) or both given in the layout fva_route writes, and then
 *          they must describe block_mask exactly.
 * softmax_scale: <= 0 selects 1/sqrt(128).
 * flags: FVA_SCHED_PERSISTENT or FVA_SCHED_NAIVE, optionally | FVA_TRACE,
 *        | FVA_SCHED_UNPAIRED and | FVA_SPLIT_BLOCKS(s). A split row's chunks
 *        run as separate work items; their partial results (fp32) are merged
 *        in chunk order, so results stay deterministic. kv_idx rows are
 *        taken in ascending order without repeats (as fva_route writes them):
 *        a paired row is processed in that order whatever order it is given.
 * O: bf16, same strides as Q; every real token row is written.
 * trace: device int64 [fva_trace_words] when FVA_TRACE is set, else ignored.
 *        Row r = (b*heads + h)*nb + i gets {start, end, (xcc_id << 16) |
 *        hw_id low bits, shader-clock cycles} (unwritten for a split row;
 *        the two rows of a pair share their item's time, half each),
 *        chunk c of a split row the same at batch*heads*nb + c (c < 2048);
 *        start and end are the 100 MHz constant device clock, the last word
 *        the item's elapsed engine-clock cycles (s_memtime), so that
 *        cycles * 100 MHz / (end - start) is the engine clock it ran at.
 */
fva_status fva_attn(const void* Q, const void* K, const void* V, const fva_qkv_desc* desc,
                    const fva_tiling* tiling, const uint8_t* block_mask, const int32_t* counts,
                    const int32_t* kv_idx, float softmax_scale, uint32_t flags, void* O, void* workspace,
                    size_t workspace_bytes, void* trace, void* stream);

/*
 * Hilbert-curve block organisation (§3.1, routing frontend: blocks are
 * reordered along a Hilbert curve so that tokens that are close in the
 * latent video land in nearby blocks at every scale).
 *
 * The curve is J. Skilling's 3D Hilbert curve ("Programming the Hilbert
 * curve", AIP Conf. Proc. 707, 2004) on the cube of side 2^k, k the smallest
 * integer with 2^k >= max(T, H, W); token (t, y, x) is the point with axes
 * (0, 1, 2) = (t, y, x), axis 0 giving the most significant bit of each
 * 3-bit digit of the curve index. The rank of a token is the number of grid
 * tokens with a smaller curve index.
 *
 * Curve layout: a curve-ordered tensor holds at sequence position r the
 * token whose rank is r. fva_route and fva_attn run on curve-ordered Q, K, V
 * with the one-dimensional tiling {T = 1, H = 1, W = N, bt = 1, bh = 1,
 * bw = B}, B in {64, 128}: block i is ranks [iB, min((i+1)B, N)), every
 * block full except the last, and O comes back curve-ordered. Permuting
 * once into curve order and once back is the caller's choice of where in
 * its model to do it (e.g. around the whole stack of attention layers).
 */
#define FVA_TO_CURVE 0   /* dst[.., r, :] = src[.., perm[r], :] */
#define FVA_FROM_CURVE 1 /* dst[.., perm[r], :] = src[.., r, :] */

/* Workspace bytes of fva_curve_order: a bitmap of 8^k bits and its word
 * prefix sums (each max(1, 8^k / 32) * 4 bytes) and one uint32 curve index
 * per token, each part 256-byte aligned. FVA_ERR_SHAPE for a non-positive
 * extent, FVA_ERR_UNSUPPORTED for an extent above 256. Host only. */
fva_status fva_curve_workspace_size(int32_t T, int32_t H, int32_t W, size_t* bytes);

/*
 * fva_curve_order -- perm[r] = raster token id (t*H + y)*W + x of the token
 * of rank r, for every r < T*H*W (device int32 [T*H*W], fully written).
 * Exact integer work; the result depends only on (T, H, W), so a caller
 * builds it once per grid and keeps it.
 * workspace: at least fva_curve_workspace_size bytes of device memory,
 *            256-byte aligned; its contents are scratch.
 * Errors as for fva_curve_workspace_size, FVA_ERR_INVALID_ARG for a NULL
 * perm, FVA_ERR_WORKSPACE for a missing or short workspace.
 */
fva_status fva_curve_order(int32_t T, int32_t H, int32_t W, int32_t* perm, void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * fva_permute_tokens -- moves whole token rows of a bf16 tensor with the
 * layout of fva_qkv_desc (head_dim 128) between raster and curve order:
 * FVA_TO_CURVE gathers dst[b,h,r,:] = src[b,h,perm[r],:], FVA_FROM_CURVE
 * scatters dst[b,h,perm[r],:] = src[b,h,r,:], for r < desc->tokens, with
 * perm from fva_curve_order (any permutation of 0 .. tokens-1 works). src
 * and dst share desc's strides and must not overlap (src == dst is
 * rejected; a partial overlap is not detected). A perm entry outside
 * [0, tokens) is never dereferenced: the gathered row is written as zeros,
 * the scattered row is dropped.
 * Errors: FVA_ERR_INVALID_ARG (NULL pointer, src == dst, rows not 16-byte
 * aligned, bad direction), FVA_ERR_SHAPE (bad extents or strides),
 * FVA_ERR_UNSUPPORTED (head_dim != 128, batch*heads > 65535).
 */
fva_status fva_permute_tokens(const void* src, void* dst, const fva_qkv_desc* desc, const int32_t* perm,
                              int32_t direction, void* stream);

/*
 * FP8 (E4M3) quantised-V attention (§3.4: V is quantised on the GPU before
 * attention on every step; the format is not named there).
 *
 * Format: OCP E4M3 (bias 7, largest finite 448, subnormals m * 2^-9),
 * round to nearest even. Every (batch, head, channel d) has a power-of-two
 * scale 2^e_d, e_d = max(-127, min{e : amax_d * 2^-e <= 448}) with
 * amax_d = max over the head's tokens of |V[., d]|, and the code of V[n, d]
 * is E4M3(V[n, d] * 2^-e_d) (exact scaling, one rounding).
 *
 * V8 layout (one 16 KB tile per block): uint8 [batch, heads, nb, 128 d,
 * 128 p]; byte (d, p) of block j holds channel d of the block's real key
 * number kap(p) (keys numbered as the tiling packs them: local raster order
 * of a box, consecutive positions of a one-dimensional block) with
 *   p = 32 g + 16 hb + 4 t + r (g, t in 0..3; hb in 0..1; r in 0..3),
 *   kap(p) = 64 hb + 32 (t / 2) + 8 g + 4 (t % 2) + r,
 * and 0 where kap(p) is past the block's real keys. v_exp: int32
 * [batch, heads, 128] = e_d.
 */
/* Bytes of the V8 tensor for this shape (batch*heads*nb*16384). Host only. */
fva_status fva_v8_size(const fva_qkv_desc* desc, const fva_tiling* tiling, size_t* bytes);

/* Workspace bytes of fva_quantize_v: one uint32 per (batch, head, channel),
 * 256-byte aligned. Host only. */
fva_status fva_quantize_v_workspace_size(const fva_qkv_desc* desc, const fva_tiling* tiling, size_t* bytes);

/*
 * fva_quantize_v -- V (bf16, desc's layout) to V8 and v_exp as above; both
 * outputs fully written (V8 16-byte aligned, v_exp 4-byte aligned).
 * Deterministic: the codes are the format's rounding, bit for bit.
 * Errors as for fva_route (shape, alignment, workspace), and
 * FVA_ERR_UNSUPPORTED for batch*heads > 65535.
 */
fva_status fva_quantize_v(const void* V, const fva_qkv_desc* desc, const fva_tiling* tiling, uint8_t* V8,
                          int32_t* v_exp, void* workspace, size_t workspace_bytes, void* stream);

/*
 * fva_attn_fp8v -- fva_attn with V replaced by its E4M3 quantisation (V8,
 * v_exp from fva_quantize_v with the same desc and tiling). Q K^T and the
 * online softmax are as in fva_attn; the probabilities of each kept block
 * are rounded to E4M3 (as P * 2^7, relative error <= 2^-4 in the format's
 * normal range, values below about 2^-17 of the row's running maximum
 * flush to zero) and multiplied with V8 on the fp8 matrix unit (fp32
 * accumulation), the V and P scales entering as the MFMA's power-of-two
 * block scales. The softmax denominator is the sum of the same rounded
 * probabilities. Flags, counts/kv_idx, workspace (fva_attn_workspace_size),
 * trace and O are as for fva_attn.
 */
fva_status fva_attn_fp8v(const void* Q, const void* K, const uint8_t* V8, const int32_t* v_exp,
                         const fva_qkv_desc* desc, const fva_tiling* tiling, const uint8_t* block_mask,
                         const int32_t* counts, const int32_t* kv_idx, float softmax_scale, uint32_t flags, void* O,
                         void* workspace, size_t workspace_bytes, void* trace, void* stream);

/*
 * Allocation-free attention, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): fva_attn with the persistent scheduler, whose work list, plan
 * scratch and block records live in a static device array of the library
 * (16 MiB on every device the library runs on, held until the process
 * ends) instead of a caller workspace. The call allocates nothing.
 *
 * Differences from fva_attn: counts and kv_idx are required (in the layout
 * fva_route writes; the mask itself is not read); flags may hold FVA_TRACE
 * only (FVA_SCHED_NAIVE, FVA_SCHED_UNPAIRED and FVA_SPLIT_BLOCKS are
 * rejected); every query block runs as its own item (no query-block pairs,
 * whose union lists are not kept; pairing changes no output bit); no row is
 * split into chunks, so where fva_attn's automatic chunk size would split rows
 * (few rows per workgroup slot) the output can differ from fva_attn's in the
 * last bits (the same sums in another order); everywhere else it is
 * identical. Inputs, O, trace and errors as for fva_attn.
 *
 * A shape needs, of the 16 MiB, the queue items (4 bytes per query block),
 * two per-row prefixes (8 bytes per query block + 8), 76 bytes per head,
 * 32 bytes per block of the tiling and 80 bytes of queue bookkeeping, each
 * part rounded up to 256 bytes: with nb = 660 about 2,000 heads fit. A
 * shape needing more returns FVA_ERR_SCRATCH before anything is launched.
 * Every call on one device shares that
 * device's scratch, and the plan kernel rewrites all of it on every call:
 * calls that overlap on one device (different streams, or host threads)
 * race and give undefined results; calls in one stream order are safe.
 */
fva_status fva_attn_noalloc(const void* Q, const void* K, const void* V, const fva_qkv_desc* desc,
                            const fva_tiling* tiling, const int32_t* counts, const int32_t* kv_idx,
                            float softmax_scale, uint32_t flags, void* O, void* trace, void* stream);

/* Static description of a status code. */
const char* fva_status_string(fva_status status);

#ifdef __cplusplus
}
#endif

#endif /* FVA_H */
