// C ABI of libpsa (declared in include/psa.h): argument validation, workspace layout and
// kernel dispatch.  All device work lives in psa_kernels.hip.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>

#include "psa_launch.h"

namespace {

thread_local char g_error[512] = "";

psa_status_t fail(psa_status_t status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_error, sizeof(g_error), fmt, ap);
  va_end(ap);
  return status;
}

// Restores the thread's error detail when it goes out of scope.
struct SavedError {
  char text[sizeof(g_error)];
  SavedError() { memcpy(text, g_error, sizeof(text)); }
  ~SavedError() { memcpy(g_error, text, sizeof(text)); }
};

psa_status_t hip_fail(hipError_t e, const char* what) {
  return fail(PSA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Token and block counts of a grid; false if the grid is invalid or too large for int32 indices.
bool grid_geometry(psa_grid_t grid, int32_t block, psa::Geometry* g) {
  if (grid.frames < 1 || grid.height < 1 || grid.width < 1 || grid.n_text < 0 || block < 1)
    return false;
  const int64_t hw = (int64_t)grid.height * grid.width;
  const int64_t n_video = hw * grid.frames;
  const int64_t n = n_video + grid.n_text;
  if (n + 2 * (int64_t)block >= ((int64_t)1 << 31)) return false;
  *g = psa::Geometry{};
  g->hw = (int32_t)hw;
  g->n_video = (int32_t)n_video;
  g->n = (int32_t)n;
  g->n_text = grid.n_text;
  g->block = block;
  g->nb = (int32_t)((n + block - 1) / block);
  g->frames = grid.frames;
  g->height = grid.height;
  g->width = grid.width;
  return true;
}

// Geometry of the PSABlock-centric layout (3D padding, Sec. 3.2) cut into tiles of `tile`
// positions; tile = 0 only sizes the layout (PSABlock-level maps).
psa_status_t geometry_3d(psa_grid_t grid, psa_block3d_t pb, int32_t tile, psa::Geometry* g) {
  if (grid.frames < 1 || grid.height < 1 || grid.width < 1 || grid.n_text < 0)
    return fail(PSA_ERR_INVALID, "invalid grid (%d x %d x %d + %d text)", grid.frames, grid.height,
                grid.width, grid.n_text);
  if (pb.t < 1 || pb.h < 1 || pb.w < 1)
    return fail(PSA_ERR_INVALID, "PSABlock sizes must be >= 1 (got %d x %d x %d)", pb.t, pb.h, pb.w);
  const int64_t tp = (grid.frames + (int64_t)pb.t - 1) / pb.t;
  const int64_t hp = (grid.height + (int64_t)pb.h - 1) / pb.h;
  const int64_t wp = (grid.width + (int64_t)pb.w - 1) / pb.w;
  const int64_t vol = (int64_t)pb.t * pb.h * pb.w;
  const int64_t n_blk = tp * hp * wp * vol;
  const int64_t n = n_blk + grid.n_text;
  const int64_t n_video = (int64_t)grid.frames * grid.height * grid.width;
  if (vol >= ((int64_t)1 << 31) || n + 256 >= ((int64_t)1 << 31) || n_video + grid.n_text + 256 >= ((int64_t)1 << 31))
    return fail(PSA_ERR_UNSUPPORTED, "PSABlock layout of %lld tokens is too large", (long long)n);
  if (tile != 0 && vol % tile != 0)
    return fail(PSA_ERR_UNSUPPORTED, "a PSABlock of %lld tokens is not a whole number of %d-token tiles",
                (long long)vol, tile);
  *g = psa::Geometry{};
  g->hw = grid.height * grid.width;
  g->n_video = (int32_t)n_video;
  g->n = (int32_t)n;
  g->n_text = grid.n_text;
  g->block = tile;
  g->nb = tile ? (int32_t)((n + tile - 1) / tile) : 0;
  g->frames = grid.frames;
  g->height = grid.height;
  g->width = grid.width;
  g->pbt = pb.t;
  g->pbh = pb.h;
  g->pbw = pb.w;
  g->tp = (int32_t)tp;
  g->hp = (int32_t)hp;
  g->wp = (int32_t)wp;
  g->n_blk = (int32_t)n_blk;
  return PSA_OK;
}

// Alignment of a device pointer (NULL passes: optional outputs are checked for presence
// separately).
bool aligned(const void* p, uintptr_t bytes) { return ((uintptr_t)p & (bytes - 1)) == 0; }

// The tensors of an attention call: q, k, v and o present and 16-byte aligned (the kernels load
// and store 16-byte vectors), lse (optional) 4-byte aligned.
psa_status_t check_tensors(const void* q, const void* k, const void* v, const void* o,
                           const float* lse) {
  if (!q || !k || !v || !o) return fail(PSA_ERR_INVALID, "q, k, v and o must be non-NULL");
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16))
    return fail(PSA_ERR_INVALID, "q, k, v and o must be 16-byte aligned (%p %p %p %p)", q, k, v, o);
  if (!aligned(lse, 4)) return fail(PSA_ERR_INVALID, "lse must be 4-byte aligned (%p)", (const void*)lse);
  return PSA_OK;
}

// Optional count outputs of the map and plan calls.
psa_status_t check_counts_out(const int32_t* per_row, const int64_t* per_head) {
  if (!aligned(per_row, 4)) return fail(PSA_ERR_INVALID, "kept_per_row must be 4-byte aligned");
  if (!aligned(per_head, 8)) return fail(PSA_ERR_INVALID, "kept_per_head must be 8-byte aligned");
  return PSA_OK;
}

psa_status_t check_params(const psa_stripe_t* params, int32_t n_heads) {
  if (!params) return fail(PSA_ERR_INVALID, "params is NULL");
  if (n_heads < 1) return fail(PSA_ERR_INVALID, "n_heads must be >= 1 (got %d)", n_heads);
  for (int32_t h = 0; h < n_heads; h++) {
    const psa_stripe_t& m = params[h];
    if (m.t_w < 1 || m.s_w < 1)
      return fail(PSA_ERR_INVALID, "head %d: widths must be >= 1 (T_w=%d, S_w=%d)", h, m.t_w, m.s_w);
    if (m.t_s < 1 || m.s_s < 1)
      return fail(PSA_ERR_INVALID, "head %d: strides must be >= 1 (T_s=%d, S_s=%d)", h, m.t_s, m.s_s);
    if (m.t_o > PSA_MAX_OFFSET || m.t_o < -PSA_MAX_OFFSET || m.s_o > PSA_MAX_OFFSET ||
        m.s_o < -PSA_MAX_OFFSET)
      return fail(PSA_ERR_INVALID, "head %d: |offset| must be <= %d", h, PSA_MAX_OFFSET);
  }
  return PSA_OK;
}

psa::ParamChunk chunk_of(const psa_stripe_t* params, int32_t head0, int32_t n_heads) {
  psa::ParamChunk pc;
  pc.n = std::min(psa::kHeadsPerChunk, n_heads - head0);
  for (int32_t i = 0; i < psa::kHeadsPerChunk; i++) pc.m[i] = i < pc.n ? params[head0 + i] : params[head0];
  return pc;
}

psa_status_t check_attention_shape(int32_t batch, int32_t n_heads, int32_t head_dim,
                                   int32_t block) {
  if (batch < 1) return fail(PSA_ERR_INVALID, "batch must be >= 1 (got %d)", batch);
  if (n_heads < 1) return fail(PSA_ERR_INVALID, "n_heads must be >= 1 (got %d)", n_heads);
  if (head_dim != 64 && head_dim != 128)
    return fail(PSA_ERR_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", head_dim);
  if (block != 64 && block != 128)
    return fail(PSA_ERR_UNSUPPORTED, "block must be 64 or 128 (got %d)", block);
  return PSA_OK;
}

// Limits of the scheduler, shared by the plans and runs of both layouts.
psa_status_t check_limits(int32_t batch, int32_t n_heads, const psa::Geometry* g) {
  if (g->nb > PSA_MAX_BLOCKS)
    return fail(PSA_ERR_UNSUPPORTED, "%d blocks per sequence exceed %d", g->nb, PSA_MAX_BLOCKS);
  if ((int64_t)batch * n_heads > PSA_MAX_BATCH_HEADS)
    return fail(PSA_ERR_UNSUPPORTED, "batch*n_heads = %lld exceeds %d", (long long)batch * n_heads,
                PSA_MAX_BATCH_HEADS);
  if ((int64_t)batch * n_heads * g->nb >= ((int64_t)1 << 31))
    return fail(PSA_ERR_UNSUPPORTED, "too many work items");
  return PSA_OK;
}

// Limits of the scheduler and the workspace, shared by the plans and runs of both layouts.
psa_status_t check_work(int32_t batch, int32_t n_heads, const void* workspace,
                        size_t workspace_bytes, const psa::Geometry* g, psa::WorkspaceLayout* wl) {
  const psa_status_t s = check_limits(batch, n_heads, g);
  if (s != PSA_OK) return s;
  *wl = psa::workspace_layout(batch, n_heads, g->nb, g->pbt > 0);
  if (!workspace || workspace_bytes < wl->total)
    return fail(PSA_ERR_WORKSPACE, "workspace of %zu bytes at %p; %zu bytes required", workspace_bytes,
                workspace, wl->total);
  if (((uintptr_t)workspace & 255) != 0)
    return fail(PSA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return PSA_OK;
}

psa_status_t check_counts(int32_t batch, int32_t n_heads) {
  if (batch < 1) return fail(PSA_ERR_INVALID, "batch must be >= 1 (got %d)", batch);
  if (n_heads < 1) return fail(PSA_ERR_INVALID, "n_heads must be >= 1 (got %d)", n_heads);
  return PSA_OK;
}

// Sizes shared by the plan and the run of one-dimensional blocks.
psa_status_t check_plan(int32_t batch, int32_t n_heads, psa_grid_t grid, int32_t block,
                        const void* workspace, size_t workspace_bytes, psa::Geometry* g,
                        psa::WorkspaceLayout* wl) {
  psa_status_t s = check_counts(batch, n_heads);
  if (s != PSA_OK) return s;
  if (block != 64 && block != 128)
    return fail(PSA_ERR_UNSUPPORTED, "block must be 64 or 128 (got %d)", block);
  if (!grid_geometry(grid, block, g))
    return fail(PSA_ERR_INVALID, "invalid grid (%d x %d x %d + %d text)", grid.frames, grid.height,
                grid.width, grid.n_text);
  return check_work(batch, n_heads, workspace, workspace_bytes, g, wl);
}

// Sizes shared by the plan and the run of the PSABlock-centric layout.
psa_status_t check_plan_3d(int32_t batch, int32_t n_heads, psa_grid_t grid, psa_block3d_t pb,
                           int32_t tile, const void* workspace, size_t workspace_bytes,
                           psa::Geometry* g, psa::WorkspaceLayout* wl) {
  psa_status_t s = check_counts(batch, n_heads);
  if (s != PSA_OK) return s;
  if (tile != 64 && tile != 128)
    return fail(PSA_ERR_UNSUPPORTED, "tile must be 64 or 128 (got %d)", tile);
  s = geometry_3d(grid, pb, tile, g);
  if (s != PSA_OK) return s;
  return check_work(batch, n_heads, workspace, workspace_bytes, g, wl);
}

// Setup and schedule kernels of a plan over geometry g.
psa_status_t enqueue_plan(int32_t batch, int32_t n_heads, const psa::Geometry& g,
                          const psa_stripe_t* params, void* workspace,
                          const psa::WorkspaceLayout& wl, int32_t* kept_per_row,
                          hipStream_t stream, const char* who) {
  for (int32_t h0 = 0; h0 < n_heads; h0 += psa::kHeadsPerChunk) {
    const psa::ParamChunk pc = chunk_of(params, h0, n_heads);
    hipError_t e = psa::launch_setup(pc, h0, g, workspace, wl, h0 == 0, stream);
    if (e != hipSuccess) return hip_fail(e, who);
  }
  hipError_t e = psa::launch_schedule(g, batch, n_heads, workspace, wl, kept_per_row, stream);
  if (e != hipSuccess) return hip_fail(e, who);
  return PSA_OK;
}

psa_status_t check_layout_args(const void* a, const void* b, int32_t n_bh, int32_t head_dim) {
  if (!a || !b) return fail(PSA_ERR_INVALID, "tensors must be non-NULL");
  if (!aligned(a, 16) || !aligned(b, 16))
    return fail(PSA_ERR_INVALID, "tensors must be 16-byte aligned (%p %p)", a, b);
  if (n_bh < 1) return fail(PSA_ERR_INVALID, "batch_heads must be >= 1 (got %d)", n_bh);
  if (n_bh > 65535) return fail(PSA_ERR_UNSUPPORTED, "batch_heads must be <= 65535 (got %d)", n_bh);
  if (head_dim != 64 && head_dim != 128)
    return fail(PSA_ERR_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", head_dim);
  return PSA_OK;
}

int32_t persistent_workgroups() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return 256;
  // Two 4-wave workgroups per CU for the one-row engine (about 80 KB of LDS each); the pair engine
  // (block 128) launches half as many 8-wave workgroups, one per CU.
  return 2 * cus;
}

// The run of a plan; `rearm` = false right after the plan's own kernels, which leave the queue
// counters at zero.
psa_status_t run_planned(const void* q, const void* k, const void* v, void* o, int32_t batch,
                         int32_t n_heads, int32_t head_dim, psa_grid_t grid, int32_t block,
                         float softmax_scale, void* workspace, size_t workspace_bytes, float* lse,
                         hipStream_t stream, bool rearm) {
  psa_status_t s = check_tensors(q, k, v, o, lse);
  if (s != PSA_OK) return s;
  s = check_attention_shape(batch, n_heads, head_dim, block);
  if (s != PSA_OK) return s;
  psa::Geometry g;
  psa::WorkspaceLayout wl;
  s = check_plan(batch, n_heads, grid, block, workspace, workspace_bytes, &g, &wl);
  if (s != PSA_OK) return s;
  const float c = softmax_scale * 1.4426950408889634f;
  hipError_t e = psa::launch_sparse(q, k, v, o, lse, batch, n_heads, head_dim, g, c, workspace, wl,
                                    persistent_workgroups(), stream, rearm);
  if (e != hipSuccess) return hip_fail(e, "psa_attention_run kernel launch");
  return PSA_OK;
}

}  // namespace

extern "C" {

int32_t psa_num_blocks(psa_grid_t grid, int32_t block) {
  psa::Geometry g;
  return grid_geometry(grid, block, &g) ? g.nb : -1;
}

size_t psa_workspace_size(int32_t batch, int32_t n_heads, psa_grid_t grid, int32_t block) {
  psa::Geometry g;
  if (batch < 1 || n_heads < 1 || !grid_geometry(grid, block, &g)) return 0;
  return psa::workspace_layout(batch, n_heads, g.nb, false).total;
}

int64_t psa_blocked_tokens(psa_grid_t grid, psa_block3d_t pb) {
  psa::Geometry g;
  const SavedError keep;  // a size query leaves the error detail alone
  const psa_status_t s = geometry_3d(grid, pb, 0, &g);
  return s == PSA_OK ? (int64_t)g.n : -1;
}

psa_status_t psa_to_blocks(const void* x, void* xb, int32_t batch_heads, int32_t head_dim,
                           psa_grid_t grid, psa_block3d_t pb, hipStream_t stream) {
  psa_status_t s = check_layout_args(x, xb, batch_heads, head_dim);
  if (s != PSA_OK) return s;
  psa::Geometry g;
  s = geometry_3d(grid, pb, 0, &g);
  if (s != PSA_OK) return s;
  hipError_t e = psa::launch_layout(x, xb, batch_heads, head_dim, g, true, stream);
  return e == hipSuccess ? PSA_OK : hip_fail(e, "psa_to_blocks launch");
}

psa_status_t psa_from_blocks(const void* xb, void* x, int32_t batch_heads, int32_t head_dim,
                             psa_grid_t grid, psa_block3d_t pb, hipStream_t stream) {
  psa_status_t s = check_layout_args(xb, x, batch_heads, head_dim);
  if (s != PSA_OK) return s;
  psa::Geometry g;
  s = geometry_3d(grid, pb, 0, &g);
  if (s != PSA_OK) return s;
  hipError_t e = psa::launch_layout(xb, x, batch_heads, head_dim, g, false, stream);
  return e == hipSuccess ? PSA_OK : hip_fail(e, "psa_from_blocks launch");
}

psa_status_t psa_build_blockmap_3d(const psa_stripe_t* params, int32_t n_heads, psa_grid_t grid,
                                   psa_block3d_t pb, uint8_t* blockmap, int32_t* kept_per_row,
                                   int64_t* kept_per_head, hipStream_t stream) {
  psa::Geometry g;
  psa_status_t s = geometry_3d(grid, pb, 0, &g);
  if (s != PSA_OK) return s;
  s = check_params(params, n_heads);
  if (s != PSA_OK) return s;
  s = check_counts_out(kept_per_row, kept_per_head);
  if (s != PSA_OK) return s;
  const int64_t groups = (int64_t)g.tp * g.hp * g.wp + (grid.n_text > 0 ? 1 : 0);
  if (groups * groups >= ((int64_t)1 << 40) || groups >= ((int64_t)1 << 31))
    return fail(PSA_ERR_UNSUPPORTED, "PSABlock map of %lld groups is too large", (long long)groups);
  g.nb = (int32_t)groups;
  for (int32_t h0 = 0; h0 < n_heads; h0 += psa::kHeadsPerChunk) {
    const psa::ParamChunk pc = chunk_of(params, h0, n_heads);
    hipError_t e = psa::launch_group_blockmap(pc, h0, g, blockmap, kept_per_row, kept_per_head, stream);
    if (e != hipSuccess) return hip_fail(e, "psa_build_blockmap_3d launch");
  }
  return PSA_OK;
}

size_t psa_workspace_size_3d(int32_t batch, int32_t n_heads, psa_grid_t grid, psa_block3d_t pb,
                             int32_t tile) {
  psa::Geometry g;
  const SavedError keep;
  const psa_status_t s = (tile == 64 || tile == 128) ? geometry_3d(grid, pb, tile, &g) : PSA_ERR_UNSUPPORTED;
  if (batch < 1 || n_heads < 1 || s != PSA_OK) return 0;
  return psa::workspace_layout(batch, n_heads, g.nb, true).total;
}

psa_status_t psa_attention_plan_3d(int32_t batch, int32_t n_heads, psa_grid_t grid,
                                   psa_block3d_t pb, int32_t tile, const psa_stripe_t* params,
                                   void* workspace, size_t workspace_bytes,
                                   int32_t* kept_per_tile, hipStream_t stream) {
  psa::Geometry g;
  psa::WorkspaceLayout wl;
  psa_status_t s = check_plan_3d(batch, n_heads, grid, pb, tile, workspace, workspace_bytes, &g, &wl);
  if (s != PSA_OK) return s;
  s = check_params(params, n_heads);
  if (s != PSA_OK) return s;
  s = check_counts_out(kept_per_tile, nullptr);
  if (s != PSA_OK) return s;
  return enqueue_plan(batch, n_heads, g, params, workspace, wl, kept_per_tile, stream,
                      "psa_attention_plan_3d launch");
}

psa_status_t psa_attention_run_3d(const void* q, const void* k, const void* v, void* o,
                                  int32_t batch, int32_t n_heads, int32_t head_dim,
                                  psa_grid_t grid, psa_block3d_t pb, int32_t tile,
                                  float softmax_scale, void* workspace, size_t workspace_bytes,
                                  float* lse, hipStream_t stream) {
  psa_status_t s = check_tensors(q, k, v, o, lse);
  if (s != PSA_OK) return s;
  s = check_attention_shape(batch, n_heads, head_dim, tile);
  if (s != PSA_OK) return s;
  psa::Geometry g;
  psa::WorkspaceLayout wl;
  s = check_plan_3d(batch, n_heads, grid, pb, tile, workspace, workspace_bytes, &g, &wl);
  if (s != PSA_OK) return s;
  const float c = softmax_scale * 1.4426950408889634f;
  hipError_t e = psa::launch_sparse(q, k, v, o, lse, batch, n_heads, head_dim, g, c, workspace, wl,
                                    persistent_workgroups(), stream);
  if (e != hipSuccess) return hip_fail(e, "psa_attention_run_3d kernel launch");
  return PSA_OK;
}

psa_status_t psa_build_blockmap(const psa_stripe_t* params, int32_t n_heads, psa_grid_t grid,
                                int32_t block, uint8_t* blockmap, int32_t* kept_per_row,
                                int64_t* kept_per_head, hipStream_t stream) {
  psa::Geometry g;
  if (!grid_geometry(grid, block, &g))
    return fail(PSA_ERR_INVALID, "invalid grid (%d x %d x %d + %d text) or block %d", grid.frames,
                grid.height, grid.width, grid.n_text, block);
  psa_status_t s = check_params(params, n_heads);
  if (s != PSA_OK) return s;
  s = check_counts_out(kept_per_row, kept_per_head);
  if (s != PSA_OK) return s;
  if ((int64_t)g.nb * g.nb >= ((int64_t)1 << 40))
    return fail(PSA_ERR_UNSUPPORTED, "block map of %d x %d blocks is too large", g.nb, g.nb);
  for (int32_t h0 = 0; h0 < n_heads; h0 += psa::kHeadsPerChunk) {
    const psa::ParamChunk pc = chunk_of(params, h0, n_heads);
    hipError_t e = psa::launch_blockmap(pc, h0, g, blockmap, kept_per_row, kept_per_head, stream);
    if (e != hipSuccess) return hip_fail(e, "psa_build_blockmap launch");
  }
  return PSA_OK;
}

psa_status_t psa_attention_plan(int32_t batch, int32_t n_heads, psa_grid_t grid, int32_t block,
                                const psa_stripe_t* params, void* workspace,
                                size_t workspace_bytes, int32_t* kept_per_row,
                                hipStream_t stream) {
  psa::Geometry g;
  psa::WorkspaceLayout wl;
  psa_status_t s = check_plan(batch, n_heads, grid, block, workspace, workspace_bytes, &g, &wl);
  if (s != PSA_OK) return s;
  s = check_params(params, n_heads);
  if (s != PSA_OK) return s;
  s = check_counts_out(kept_per_row, nullptr);
  if (s != PSA_OK) return s;
  return enqueue_plan(batch, n_heads, g, params, workspace, wl, kept_per_row, stream,
                      "psa_attention_plan launch");
}

psa_status_t psa_attention_run(const void* q, const void* k, const void* v, void* o,
                               int32_t batch, int32_t n_heads, int32_t head_dim, psa_grid_t grid,
                               int32_t block, float softmax_scale, void* workspace,
                               size_t workspace_bytes, float* lse, hipStream_t stream) {
  return run_planned(q, k, v, o, batch, n_heads, head_dim, grid, block, softmax_scale, workspace,
                     workspace_bytes, lse, stream, true);
}

psa_status_t psa_attention_fwd(const void* q, const void* k, const void* v, void* o,
                               int32_t batch, int32_t n_heads, int32_t head_dim, psa_grid_t grid,
                               int32_t block, const psa_stripe_t* params, float softmax_scale,
                               void* workspace, size_t workspace_bytes, float* lse,
                               int32_t* kept_per_row, hipStream_t stream) {
  psa_status_t s = check_tensors(q, k, v, o, lse);
  if (s != PSA_OK) return s;
  s = check_attention_shape(batch, n_heads, head_dim, block);
  if (s != PSA_OK) return s;
  s = psa_attention_plan(batch, n_heads, grid, block, params, workspace, workspace_bytes,
                         kept_per_row, stream);
  if (s != PSA_OK) return s;
  return run_planned(q, k, v, o, batch, n_heads, head_dim, grid, block, softmax_scale, workspace,
                     workspace_bytes, lse, stream, false);
}

psa_status_t psa_attention_fwd_noalloc(const void* q, const void* k, const void* v, void* o,
                                       int32_t batch, int32_t n_heads, int32_t head_dim,
                                       psa_grid_t grid, int32_t block, const psa_stripe_t* params,
                                       float softmax_scale, float* lse, int32_t* kept_per_row,
                                       hipStream_t stream) {
  // Everything is validated before the first HIP call.
  psa_status_t s = check_tensors(q, k, v, o, lse);
  if (s != PSA_OK) return s;
  s = check_attention_shape(batch, n_heads, head_dim, block);
  if (s != PSA_OK) return s;
  psa::Geometry g;
  if (!grid_geometry(grid, block, &g))
    return fail(PSA_ERR_INVALID, "invalid grid (%d x %d x %d + %d text)", grid.frames, grid.height,
                grid.width, grid.n_text);
  s = check_limits(batch, n_heads, &g);
  if (s != PSA_OK) return s;
  s = check_params(params, n_heads);
  if (s != PSA_OK) return s;
  s = check_counts_out(kept_per_row, nullptr);
  if (s != PSA_OK) return s;
  const size_t need = psa::workspace_layout(batch, n_heads, g.nb, false).total;
  if (need > PSA_NOALLOC_SCRATCH_BYTES)
    return fail(PSA_ERR_WORKSPACE, "the plan of these sizes needs %zu bytes; the static scratch holds %zu",
                need, (size_t)PSA_NOALLOC_SCRATCH_BYTES);
  void* scratch = nullptr;
  const hipError_t e = psa::scratch_pointer(&scratch);
  if (e != hipSuccess) return hip_fail(e, "psa_attention_fwd_noalloc: address of the static scratch");
  return psa_attention_fwd(q, k, v, o, batch, n_heads, head_dim, grid, block, params, softmax_scale,
                           scratch, PSA_NOALLOC_SCRATCH_BYTES, lse, kept_per_row, stream);
}

size_t psa_dense_workspace_size(void) { return psa::kDenseWorkspaceBytes; }

psa_status_t psa_dense_fwd(const void* q, const void* k, const void* v, void* o, int32_t batch,
                           int32_t n_heads, int32_t head_dim, int32_t n_tokens, int32_t block,
                           float softmax_scale, float* lse, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  psa_status_t s = check_tensors(q, k, v, o, lse);
  if (s != PSA_OK) return s;
  s = check_attention_shape(batch, n_heads, head_dim, block);
  if (s != PSA_OK) return s;
  if (n_tokens < 1 || (int64_t)n_tokens + 2 * block >= ((int64_t)1 << 31))
    return fail(PSA_ERR_INVALID, "n_tokens must be in [1, 2^31 - 2*block) (got %d)", n_tokens);
  const int64_t items = (int64_t)batch * n_heads * ((n_tokens + block - 1) / block);
  if (items + 8 >= ((int64_t)1 << 31)) return fail(PSA_ERR_UNSUPPORTED, "too many work items");
  if (workspace && workspace_bytes < psa::kDenseWorkspaceBytes)
    return fail(PSA_ERR_WORKSPACE, "dense workspace of %zu bytes; %zu bytes required", workspace_bytes,
                psa::kDenseWorkspaceBytes);
  if (((uintptr_t)workspace & 255) != 0)
    return fail(PSA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  const float c = softmax_scale * 1.4426950408889634f;
  hipError_t e = psa::launch_dense(q, k, v, o, lse, batch, n_heads, head_dim, n_tokens, block, c,
                                   (int32_t*)workspace, persistent_workgroups(), stream);
  if (e != hipSuccess) return hip_fail(e, "psa_dense_fwd kernel launch");
  return PSA_OK;
}

size_t psa_l2_workspace_size(int32_t batch_heads) {
  return batch_heads < 1 ? 0 : (size_t)batch_heads * psa::kL2Chunks * 2 * sizeof(double);
}

psa_status_t psa_l2_distance(const void* o, const void* ref, int32_t batch_heads, int32_t n_tokens,
                             int32_t head_dim, double* sq_err, double* sq_ref, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  if (!o || !ref || !sq_err) return fail(PSA_ERR_INVALID, "o, ref and sq_err must be non-NULL");
  if (batch_heads < 1 || n_tokens < 1)
    return fail(PSA_ERR_INVALID, "batch_heads and n_tokens must be >= 1 (got %d, %d)", batch_heads,
                n_tokens);
  if (batch_heads > 65535)
    return fail(PSA_ERR_UNSUPPORTED, "batch_heads must be <= 65535 (got %d)", batch_heads);
  if (head_dim < 8 || head_dim % 8 != 0)
    return fail(PSA_ERR_UNSUPPORTED, "head_dim must be a positive multiple of 8 (got %d)", head_dim);
  if (!aligned(o, 16) || !aligned(ref, 16))
    return fail(PSA_ERR_INVALID, "o and ref must be 16-byte aligned");
  if (!aligned(sq_err, 8) || !aligned(sq_ref, 8))
    return fail(PSA_ERR_INVALID, "sq_err and sq_ref must be 8-byte aligned");
  if (!workspace || workspace_bytes < psa_l2_workspace_size(batch_heads))
    return fail(PSA_ERR_WORKSPACE, "workspace of %zu bytes; %zu bytes required", workspace_bytes,
                psa_l2_workspace_size(batch_heads));
  if (!aligned(workspace, 8)) return fail(PSA_ERR_WORKSPACE, "workspace must be 8-byte aligned");
  hipError_t e = psa::launch_l2(o, ref, batch_heads, (int64_t)n_tokens * head_dim, (double*)workspace,
                                sq_err, sq_ref, stream);
  return e == hipSuccess ? PSA_OK : hip_fail(e, "psa_l2_distance launch");
}

const char* psa_status_string(psa_status_t status) {
  switch (status) {
    case PSA_OK: return "PSA_OK";
    case PSA_ERR_INVALID: return "PSA_ERR_INVALID: invalid argument";
    case PSA_ERR_UNSUPPORTED: return "PSA_ERR_UNSUPPORTED: unsupported shape";
    case PSA_ERR_WORKSPACE: return "PSA_ERR_WORKSPACE: workspace missing or too small";
    case PSA_ERR_HIP: return "PSA_ERR_HIP: HIP runtime error";
  }
  return "unknown psa_status_t";
}

const char* psa_last_error(void) { return g_error; }

}  // extern "C"
