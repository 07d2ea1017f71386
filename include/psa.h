/*
 * psa.h -- C ABI of libpsa: forward pass of PSA (Parameterized Stripe Attention) block-sparse
 * spatio-temporal attention on AMD Instinct MI355X (gfx950).
 *
 * The operation (paper: "Parameterized Stripe Attention for Efficient Video Generation"):
 *
 *  - Sec. 3.2, "Unified Representation": every attention head carries six integers
 *    M = (T_w, T_o, T_s, S_w, S_o, S_s): width, offset and stride of the inter-frame (temporal)
 *    and intra-frame (spatial) diagonal stripes.
 *  - Algorithm 1 (PSA mask definition): a query at frame t_q, in-frame position s_q may attend to
 *    a key at (t_k, s_k) iff (|t_k - t_q - T_o| mod T_s) <= T_w - 1 and
 *    (|s_k - s_q - S_o| mod S_s) <= S_w - 1.
 *  - Sec. 3.2, "Hardware-Aware Design": the test is applied per (query block, key block) pair,
 *    never per token.  Here a block is `block` consecutive tokens of the frame-major (t, h, w)
 *    sequence; its coordinates are those of its first token: t = (b*block) div (H*W),
 *    s = ((b*block) mod (H*W)) div block.  Temporal parameters therefore count frames and
 *    spatial parameters count block slots within a frame.  Text tokens appended after the
 *    F*H*W video tokens are global: a block holding any text token is kept in its whole row and
 *    column.
 *  - Algorithm 2 (PSA-Kernel): for each query block, only the kept key/value blocks are visited;
 *    S = Q K^T, keys past the end of the sequence get -inf, safe (online) softmax, O += P V.
 *
 * Conventions shared by every call:
 *  - Tensors are bf16, contiguous, layout [batch][n_heads][N][head_dim] (row-major).
 *  - Tensor pointers are device pointers owned by the caller; nothing is retained after the
 *    call.  `params` is a host array of n_heads entries, read before the call returns.
 *  - Alignment: bf16 tensors 16 bytes (the kernels move 16-byte vectors), float and int32
 *    arrays 4 bytes, int64 arrays 8 bytes; a misaligned pointer is rejected with
 *    PSA_ERR_INVALID.
 *  - Every call only enqueues work on `stream` (0 = the null stream of the current device) and
 *    returns; results are ready after the caller synchronises that stream.  The current device
 *    must be the stream's device.  What a call enqueues is kernels only (no memset, copy,
 *    allocation or synchronisation), so a caller may capture it in a HIP graph and replay it;
 *    a replay reads the buffers and, for a run, the plan the captured call was given.
 *  - Arguments are validated before anything is enqueued: on PSA_ERR_INVALID,
 *    PSA_ERR_UNSUPPORTED or PSA_ERR_WORKSPACE no output byte is written.  PSA_ERR_HIP reports a
 *    failed HIP call (launch); psa_last_error() then holds the HIP message.
 *  - The library allocates nothing and holds no mutable global state apart from the thread-local
 *    error message, the static device scratch of psa_attention_fwd_noalloc and its per-device
 *    address table; calls are re-entrant.  Two calls that share an output, a workspace or (for
 *    psa_attention_fwd_noalloc) a GPU's scratch must not overlap in time.
 *  - Numerics: q is multiplied by softmax_scale * log2(e) and rounded to bf16 once; bf16 x bf16
 *    products accumulated in fp32 (MFMA); softmax statistics in fp32 in the exp2 domain; P
 *    rounded to bf16 before P V, and the normaliser sums the rounded P; O rounded to bf16 (round
 *    to nearest even).  A query row with no kept key gets O = 0 and LSE = -inf.
 */
#ifndef PSA_H
#define PSA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Stride meaning "a single diagonal" (paper appendix on candidate initialisation: an infinite
 * stride leaves one diagonal; any stride >= the axis extent plus |offset| behaves the same). */
#define PSA_STRIDE_INF 0x7fffffff

/* Largest |offset| accepted. */
#define PSA_MAX_OFFSET (1 << 24)

/* Largest number of blocks per sequence accepted by psa_attention_fwd. */
#define PSA_MAX_BLOCKS 7936

/* Largest batch * n_heads accepted by psa_attention_fwd (scheduler limit). */
#define PSA_MAX_BATCH_HEADS 1024

/* Bytes of the static device scratch of psa_attention_fwd_noalloc, per GPU (16 MiB). */
#define PSA_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

/* M(T_w, T_o, T_s, S_w, S_o, S_s) of one head (Sec. 3.2).  Widths and strides must be >= 1. */
typedef struct {
  int32_t t_w, t_o, t_s;
  int32_t s_w, s_o, s_s;
} psa_stripe_t;

/* Latent video grid F x H x W (frame-major) followed by n_text text tokens:
 * N = frames * height * width + n_text. */
typedef struct {
  int32_t frames, height, width, n_text;
} psa_grid_t;

typedef enum {
  PSA_OK = 0,
  PSA_ERR_INVALID = 1,     /* null or misaligned pointer, width/stride < 1, |offset| too large,
                              bad sizes */
  PSA_ERR_UNSUPPORTED = 2, /* head_dim or block outside {64, 128}, too many blocks or heads */
  PSA_ERR_WORKSPACE = 3,   /* workspace NULL or smaller than psa_workspace_size() */
  PSA_ERR_HIP = 4          /* a HIP runtime call failed; see psa_last_error() */
} psa_status_t;

/* Number of blocks ceil(N / block) of the grid, or -1 if grid or block is invalid. */
int32_t psa_num_blocks(psa_grid_t grid, int32_t block);

/* Bytes of device workspace psa_attention_plan / psa_attention_fwd need for these sizes
 * (0 if invalid).  The workspace holds a plan: the per-head parameters, the block coordinates,
 * the work of every work item, the load-balanced work order, the queue counters and a header
 * naming the sizes the plan was made for; at block 128 also a signature of each query block's
 * kept set and the pairs of query blocks that form the work items. */
size_t psa_workspace_size(int32_t batch, int32_t n_heads, psa_grid_t grid, int32_t block);

/* Block map of Algorithm 1 at block granularity (Sec. 3.2), computed on the device by the same
 * decoder that psa_attention_fwd runs inside its kernels.  block >= 1 (block = 1 evaluates
 * Algorithm 1 token by token).  Any output may be NULL (not written):
 *   blockmap      device uint8 [n_heads][nb][nb]; row = query block, column = key block; 1 = kept
 *   kept_per_row  device int32 [n_heads][nb]: kept key blocks of each query block
 *   kept_per_head device int64 [n_heads]: kept tiles of each head
 * with nb = psa_num_blocks(grid, block). */
psa_status_t psa_build_blockmap(const psa_stripe_t* params, int32_t n_heads, psa_grid_t grid,
                                int32_t block, uint8_t* blockmap, int32_t* kept_per_row,
                                int64_t* kept_per_head, hipStream_t stream);

/* Plan of psa_attention_run (the work list of Algorithm 2 without the attention itself): copies
 * the stripe parameters of each head to the workspace, counts the kept key blocks of every
 * work item with the Algorithm 1 decoder and orders the items.  A work item is one (batch, head,
 * query block) at block 64; at block 128 it is a pair of query blocks of one (batch, head) that
 * share one K/V stream, the pairs formed from query blocks with equal kept sets first (the rest
 * in index order) and weighed by the union of the two sets.  Order: items
 * of more than three times the mean work (rows that keep every key block, such as text rows)
 * first, longest first, then the heads longest first, each split into equal-work ranges, one
 * work queue per XCD.  At block 128 the plan also chooses where each pair item's K/V stream
 * starts (each row still visits each of its kept blocks once, cyclically ascending from there):
 * where the item started just before it on its queue is predicted to be by then, so that the items
 * in flight on one XCD read the same key blocks at about the same time and its L2 serves them
 * once; pairs that keep every block start at block 0.  The plan
 * depends only on the sizes and on params, so one plan serves any number of runs (a layer's
 * stripes stay fixed over the denoising steps).
 *   workspace     device, psa_workspace_size(batch, n_heads, grid, block) bytes or more,
 *                 256-byte aligned; owned by the caller, overwritten
 *   kept_per_row  device int32 [n_heads][nb]: kept key blocks of each query block, or NULL
 * Limits: nb <= PSA_MAX_BLOCKS, batch * n_heads <= PSA_MAX_BATCH_HEADS, block 64 or 128. */
psa_status_t psa_attention_plan(int32_t batch, int32_t n_heads, psa_grid_t grid, int32_t block,
                                const psa_stripe_t* params, void* workspace,
                                size_t workspace_bytes, int32_t* kept_per_row,
                                hipStream_t stream);

/* Sparse attention over a planned workspace (Algorithm 2): one persistent kernel whose
 * workgroups pop work items from the plan's queues, decode the kept key blocks of each query
 * block (Algorithm 1) and run the tile engine over them.  Arguments as in psa_attention_fwd.  The
 * workspace must hold a plan made for the same batch, n_heads, grid and block; the kernel checks
 * the plan's header first and, on a mismatch or an unfinished plan, writes nothing (o and lse keep
 * their contents; no error can be returned for a condition found on the device).  The run
 * re-arms the plan's queue counters (a one-thread kernel ahead of the attention kernel) and
 * consumes them, so runs over one workspace must not overlap in time (use one workspace per
 * stream). */
psa_status_t psa_attention_run(const void* q, const void* k, const void* v, void* o,
                               int32_t batch, int32_t n_heads, int32_t head_dim, psa_grid_t grid,
                               int32_t block, float softmax_scale, void* workspace,
                               size_t workspace_bytes, float* lse, hipStream_t stream);

/* PSA block-sparse attention forward (Algorithm 2): o = softmax(scale * q k^T restricted to the
 * kept blocks of each head) v.  Equivalent to psa_attention_plan followed by psa_attention_run
 * (without the run's re-arm kernel: the plan's own kernels leave the queue counters armed).
 *   q, k, v, o     device bf16 [batch][n_heads][N][head_dim]; N = frames*height*width + n_text
 *   head_dim       64 or 128;  block: 64 or 128 (query and key block size, the tile size)
 *   params         host [n_heads]; the same M for every batch element
 *   softmax_scale  multiplies q.k before the softmax (typically 1/sqrt(head_dim))
 *   workspace      device, at least psa_workspace_size(batch, n_heads, grid, block) bytes,
 *                  256-byte aligned; contents on entry are ignored and are clobbered
 *   lse            device fp32 [batch][n_heads][N] (natural-log softmax normaliser), or NULL
 *   kept_per_row   device int32 [n_heads][nb]: the kept-block counts decoded for the schedule,
 *                  or NULL */
psa_status_t psa_attention_fwd(const void* q, const void* k, const void* v, void* o,
                               int32_t batch, int32_t n_heads, int32_t head_dim, psa_grid_t grid,
                               int32_t block, const psa_stripe_t* params, float softmax_scale,
                               void* workspace, size_t workspace_bytes, float* lse,
                               int32_t* kept_per_row, hipStream_t stream);

/* psa_attention_fwd without a workspace argument and without any allocation, for callers that
 * cannot allocate device memory: code under HIP graph capture, serving loops and harnesses that
 * forbid hipMalloc.  The plan goes to a static device array of the library instead: every GPU the
 * library runs on holds PSA_NOALLOC_SCRATCH_BYTES for it from the time the library's code is
 * loaded there until the process ends.  Arguments, result and errors as psa_attention_fwd; sizes
 * whose psa_workspace_size() exceeds PSA_NOALLOC_SCRATCH_BYTES (about 800,000 heads x blocks at
 * batch 1; 40 heads of the Wan 2.1 14B grid take 0.5 MB) are rejected with PSA_ERR_WORKSPACE before
 * anything is enqueued.  The call makes no allocation, free or copy: on the first call on a device
 * it looks up the array's address on that device (hipGetSymbolAddress), then it enqueues the
 * kernels of psa_attention_fwd.  All calls on one GPU share that GPU's array, and each leaves its
 * plan there: calls that overlap in time on one GPU (on different streams or from different host
 * threads) race and must not be made. */
psa_status_t psa_attention_fwd_noalloc(const void* q, const void* k, const void* v, void* o,
                                       int32_t batch, int32_t n_heads, int32_t head_dim,
                                       psa_grid_t grid, int32_t block, const psa_stripe_t* params,
                                       float softmax_scale, float* lse, int32_t* kept_per_row,
                                       hipStream_t stream);

/* Bytes of device workspace psa_dense_fwd can use (a constant: queue bounds and counters). */
size_t psa_dense_workspace_size(void);

/* Dense attention forward with the same tile engine (every block kept).  Sec. 4, setup: the first
 * 20 % of the denoising steps keep full attention (FlashAttention-3 in the paper's runs), and the
 * paper's kernel speedups are quoted against that full attention; this call plays both roles, the
 * attention of the steps that run dense and the speedup baseline.  Same tensor layout, with
 * N = n_tokens.  At full density psa_attention_fwd returns the same bits as this call.
 *   workspace      device, psa_dense_workspace_size() bytes or more, 256-byte aligned, or NULL.
 *                  With a workspace a small kernel arms per-XCD work queues in it and a
 *                  persistent grid takes the work items, each workgroup from its own XCD's queue
 *                  first and then from the others, so XCDs that run at different clocks finish
 *                  together.  Without one, each XCD gets an equal fixed share.  The output is
 *                  the same bits either way.  Calls sharing a workspace must not overlap in time.
 * A workspace that is too small or misaligned is rejected with PSA_ERR_WORKSPACE. */
psa_status_t psa_dense_fwd(const void* q, const void* k, const void* v, void* o, int32_t batch,
                           int32_t n_heads, int32_t head_dim, int32_t n_tokens, int32_t block,
                           float softmax_scale, float* lse, void* workspace,
                           size_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------------------------
 * 3D PSABlocks and 3D padding (Sec. 3.2, "Hardware-Aware Design" and "3D-Padding for Resolution
 * Flexibility").  A PSABlock is a bt x bh x bw tile of the F x H x W video grid; each axis is
 * padded to the smallest multiple of its block size, giving a grid of PSABlocks
 * T' = ceil(F / bt), H' = ceil(H / bh), W' = ceil(W / bw).  Algorithm 1 runs on that grid: a
 * PSABlock (t', h', w') has temporal coordinate t' and spatial coordinate h' W' + w', so
 * temporal parameters count PSABlocks along time and spatial parameters count PSABlocks of the
 * H' x W' plane.  Text tokens (after the video) are global.
 *
 * The PSABlock-centric layout of a [batch*heads][F*H*W + n_text][head_dim] tensor is
 * [batch*heads][T' H' W' bt bh bw + n_text][head_dim]: PSABlocks in row-major (t', h', w')
 * order, the tokens of each PSABlock contiguous in row-major (t, h, w) order, zeros at padded
 * positions, then the text tokens.  Attention runs on that layout in tiles of 64 or 128
 * positions (a PSABlock must be a whole number of tiles); padded keys get -inf before the
 * softmax (Algorithm 2), a tile holding only padding is never visited, and O rows at padded
 * positions are unspecified (psa_from_blocks drops them).
 * --------------------------------------------------------------------------------------------- */

/* PSABlock shape (bt, bh, bw), each >= 1. */
typedef struct {
  int32_t t, h, w;
} psa_block3d_t;

/* Positions of the PSABlock-centric layout, T' H' W' bt bh bw + n_text, or -1 if invalid. */
int64_t psa_blocked_tokens(psa_grid_t grid, psa_block3d_t pb);

/* Original -> PSABlock-centric layout (and back: psa_from_blocks, which drops padded rows).
 *   x   device bf16 [batch_heads][F*H*W + n_text][head_dim]
 *   xb  device bf16 [batch_heads][psa_blocked_tokens(grid, pb)][head_dim]
 * head_dim 64 or 128, batch_heads <= 65535.  Memory-bound copies; source and destination
 * must not overlap. */
psa_status_t psa_to_blocks(const void* x, void* xb, int32_t batch_heads, int32_t head_dim,
                           psa_grid_t grid, psa_block3d_t pb, hipStream_t stream);
psa_status_t psa_from_blocks(const void* xb, void* x, int32_t batch_heads, int32_t head_dim,
                             psa_grid_t grid, psa_block3d_t pb, hipStream_t stream);

/* Block map of Algorithm 1 at PSABlock granularity.  G = T'H'W' groups (+1: the text, last):
 *   blockmap device uint8 [n_heads][G][G], kept_per_row int32 [n_heads][G],
 *   kept_per_head int64 [n_heads]; any may be NULL. */
psa_status_t psa_build_blockmap_3d(const psa_stripe_t* params, int32_t n_heads, psa_grid_t grid,
                                   psa_block3d_t pb, uint8_t* blockmap, int32_t* kept_per_row,
                                   int64_t* kept_per_head, hipStream_t stream);

/* Workspace bytes of psa_attention_plan_3d / psa_attention_run_3d (0 if invalid); it also holds
 * the valid positions of every tile (16 bytes per tile). */
size_t psa_workspace_size_3d(int32_t batch, int32_t n_heads, psa_grid_t grid, psa_block3d_t pb,
                             int32_t tile);

/* Plan of the sparse attention over the PSABlock-centric layout, as psa_attention_plan.  The
 * work items are the tiles; kept_per_tile (device int32 [n_heads][nt], nt = ceil(
 * psa_blocked_tokens / tile), or NULL) receives the kept key tiles of every query tile (0 for a
 * tile of padding).  Limits: nt <= PSA_MAX_BLOCKS, batch * n_heads <= PSA_MAX_BATCH_HEADS. */
psa_status_t psa_attention_plan_3d(int32_t batch, int32_t n_heads, psa_grid_t grid,
                                   psa_block3d_t pb, int32_t tile, const psa_stripe_t* params,
                                   void* workspace, size_t workspace_bytes,
                                   int32_t* kept_per_tile, hipStream_t stream);

/* Sparse attention over a 3D plan, as psa_attention_run; q, k, v, o (and lse: fp32
 * [batch][n_heads][psa_blocked_tokens]) are in the PSABlock-centric layout. */
psa_status_t psa_attention_run_3d(const void* q, const void* k, const void* v, void* o,
                                  int32_t batch, int32_t n_heads, int32_t head_dim,
                                  psa_grid_t grid, psa_block3d_t pb, int32_t tile,
                                  float softmax_scale, void* workspace, size_t workspace_bytes,
                                  float* lse, hipStream_t stream);

/* ---------------------------------------------------------------------------------------------
 * PSA-Search scoring (Algorithm 3 in the appendix "Process of PSA-Search"; Sec. 3.3): the L2
 * loss between a head's sparse attention output under a candidate mask and its full attention
 * output.  A search evaluates each candidate with psa_attention_fwd (one candidate per head per
 * call) against psa_dense_fwd, and reduces both outputs here.
 * --------------------------------------------------------------------------------------------- */

/* Bytes of device workspace of psa_l2_distance (0 if batch_heads < 1). */
size_t psa_l2_workspace_size(int32_t batch_heads);

/* Per (batch, head) row r: sq_err[r] = sum over tokens and channels of (o - ref)^2 and
 * sq_ref[r] = sum of ref^2 (relative L2 loss = sqrt(sq_err / sq_ref)).  Products and sums in
 * fp32 within 64 chunks per row, combined in fp64 in a fixed order: the result is
 * deterministic.
 *   o, ref          device bf16 [batch_heads][n_tokens][head_dim], 16-byte aligned
 *   sq_err, sq_ref  device double [batch_heads] (sq_ref may be NULL)
 *   workspace       device, psa_l2_workspace_size(batch_heads) bytes, 8-byte aligned
 * head_dim a multiple of 8, batch_heads <= 65535. */
psa_status_t psa_l2_distance(const void* o, const void* ref, int32_t batch_heads, int32_t n_tokens,
                             int32_t head_dim, double* sq_err, double* sq_ref, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);

/* Static description of a status code. */
const char* psa_status_string(psa_status_t status);

/* Detail of the last non-OK status returned on the calling thread ("" if none). */
const char* psa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PSA_H */
