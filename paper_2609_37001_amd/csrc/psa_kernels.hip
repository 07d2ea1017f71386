// PSA block-sparse attention forward: HIP kernels for gfx950 (CDNA4, MI355X).
//
// Kernels
//   psa_blockmap_kernel / psa_rowcount_kernel  block map and kept counts (Algorithm 1 per block)
//   psa_setup_kernel                           stripe parameters and block coordinates -> workspace
//   psa_count_kernel                           kept key blocks of every (batch, head, query block),
//                                              and kept-set signatures for the pairing
//   psa_pairing_kernel / psa_paircount_kernel  pairs of query blocks (block 128) and their work
//   psa_schedule_kernel                        load-balanced work order split over 8 XCD queues
//   psa_starts_kernel                          block 128: where each pair item's K/V stream starts
//   psa_pair_kernel                            block 128: persistent block-sparse attention
//                                              (Algorithm 2) on pairs of query blocks, or dense
//   psa_sparse_kernel / psa_dense_kernel       block 64: the same with one query block per item
//
// Tile engine (per wave; at block 64 one workgroup of BLK/32 wave64s per query block of BLK rows
// and two workgroups per CU, at block 128 one eight-wave workgroup per CU on a pair of query
// blocks, so two waves share each SIMD either way; head dim D):
//   * every wave owns 32 query rows of the query block and all BLK keys of each key/value
//     block; lane l holds row l & 31, lanes l and l ^ 32 split its keys.  A block is processed
//     in two halves of BLK/2 keys, each with its own online-softmax update.
//   * S^T = K Q^T with v_mfma_f32_32x32x16_bf16: K rows come from LDS (A operand), Q^T stays in
//     registers (B operand).  K rows are read in a permuted order so that each lane's fp32
//     accumulators hold 8 consecutive keys of every 16-key chunk, which is exactly the B operand
//     layout of the next product: P^T needs no data movement.
//   * O^T += V^T P^T: V stays row-major in LDS and the A operand is assembled with the gfx950 LDS
//     transpose read (ds_read_b64_tr_b16).
//   * K and V fill LDS by direct global->LDS 16-byte loads (global_load_lds_dwordx4).  Block 64:
//     one K and one V buffer per workgroup, loaded by halves, each half of the next block issued
//     as soon as the last reader of that half of the current block has passed a barrier.
//     Block 128: a double buffer shared by the two query blocks of a pair, one barrier per
//     block.  16-byte chunks are XOR-swizzled per row so both the K reads and the transposed V
//     reads are bank-conflict free.
//   * Softmax in the exp2 domain: Q is multiplied by scale*log2(e) once, and the S^T
//     accumulators start at -m, so the MFMAs deliver the exponent directly; the running max is
//     raised lazily (only when a new max exceeds it by more than 8, i.e. P <= 2^8), which is
//     exact.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "psa_launch.h"

namespace psa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define PSA_LDS __attribute__((address_space(3)))

// ---------------------------------------------------------------------------------------------
// Stripe decoder: Algorithm 1 evaluated on block coordinates.
// ---------------------------------------------------------------------------------------------

// One axis of Algorithm 1: (|delta - offset| mod stride) <= width - 1.
__device__ __forceinline__ bool axis_keep(int32_t delta, int32_t width, int32_t offset,
                                          int32_t stride) {
  const int32_t x = delta - offset;
  const uint32_t ax = (uint32_t)(x < 0 ? -x : x);
  return (ax % (uint32_t)stride) < (uint32_t)width;
}

// Coordinates of block b from its first token: frame t and slot s; t = -1 marks a global block
// (a block holding at least one appended text token).
__device__ __forceinline__ int2 block_coord(const Geometry& g, int32_t b) {
  const int32_t i0 = b * g.block;
  const int32_t len = min(g.block, g.n - i0);
  if (g.n_text > 0 && i0 + len > g.n_video) return make_int2(-1, 0);
  const int32_t t = i0 / g.hw;
  return make_int2(t, (i0 - t * g.hw) / g.block);
}

// Coordinates of tile b of the PSABlock-centric layout: those of the PSABlock holding it
// (t', s' = h' W' + w'), or global for a text tile.  A PSABlock is a whole number of tiles.
__device__ __forceinline__ int2 tile_coord3d(const Geometry& g, int32_t b) {
  const int32_t i0 = b * g.block;
  if (i0 >= g.n_blk) return make_int2(-1, 0);
  const int32_t pb = i0 / (g.pbt * g.pbh * g.pbw), plane = g.hp * g.wp;
  const int32_t t = pb / plane;
  return make_int2(t, pb - t * plane);
}

// Coordinates of group i of a PSABlock-level map: PSABlock i, or the text group (global).
__device__ __forceinline__ int2 group_coord(const Geometry& g, int32_t i) {
  const int32_t plane = g.hp * g.wp;
  if (i >= g.tp * plane) return make_int2(-1, 0);
  const int32_t t = i / plane;
  return make_int2(t, i - t * plane);
}

// Whether position p of the PSABlock-centric layout holds a token (not 3D padding, not past
// the end).
__device__ __forceinline__ bool position_valid(const Geometry& g, int32_t p) {
  if (p >= g.n) return false;
  if (p >= g.n_blk) return true;
  const int32_t area = g.pbh * g.pbw, vol = g.pbt * area, plane = g.hp * g.wp;
  const int32_t pb = p / vol, x = p - pb * vol;
  const int32_t tq = pb / plane, r = pb - tq * plane, hq = r / g.wp, wq = r - hq * g.wp;
  const int32_t it = x / area, r2 = x - it * area, ih = r2 / g.pbw, iw = r2 - ih * g.pbw;
  return tq * g.pbt + it < g.frames && hq * g.pbh + ih < g.height && wq * g.pbw + iw < g.width;
}

__device__ __forceinline__ bool tile_keep(const psa_stripe_t& m, int2 q, int2 k) {
  if (q.x == kDeadTile || k.x == kDeadTile) return false;
  if (q.x < 0 || k.x < 0) return true;
  return axis_keep(k.x - q.x, m.t_w, m.t_o, m.t_s) && axis_keep(k.y - q.y, m.s_w, m.s_o, m.s_s);
}

__device__ __forceinline__ int wave_sum(int v) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// Wave-wide sum (OP 0), minimum (1) or maximum (2) in every lane, without LDS: DPP moves
// within the 16-lane rows, then the gfx950 permlane swaps across rows.
template <int OP>
__device__ __forceinline__ int32_t wave_reduce(int32_t v) {
  auto op = [](int32_t a, int32_t b) { return OP == 0 ? a + b : (OP == 1 ? min(a, b) : max(a, b)); };
  v = op(v, __builtin_amdgcn_update_dpp(v, v, 0xb1, 0xf, 0xf, false));   // quad_perm 1,0,3,2
  v = op(v, __builtin_amdgcn_update_dpp(v, v, 0x4e, 0xf, 0xf, false));   // quad_perm 2,3,0,1
  v = op(v, __builtin_amdgcn_update_dpp(v, v, 0x124, 0xf, 0xf, false));  // row_ror:4
  v = op(v, __builtin_amdgcn_update_dpp(v, v, 0x128, 0xf, 0xf, false));  // row_ror:8
  const auto r16 = __builtin_amdgcn_permlane16_swap((uint32_t)v, (uint32_t)v, false, false);
  v = op((int32_t)r16[0], (int32_t)r16[1]);                               // lanes l, l ^ 16
  const auto r32 = __builtin_amdgcn_permlane32_swap((uint32_t)v, (uint32_t)v, false, false);
  return op((int32_t)r32[0], (int32_t)r32[1]);                            // lanes l, l ^ 32
}

// Lane i receives lane i ^ m of x (m = 1, 2, 4, 8 by DPP within a 16-lane row; 16 by a shuffle).
template <int M>
__device__ __forceinline__ int32_t lane_xor(int32_t x, int lane) {
  if constexpr (M == 1) return __builtin_amdgcn_update_dpp(x, x, 0xb1, 0xf, 0xf, false);  // quad_perm 1,0,3,2
  if constexpr (M == 2) return __builtin_amdgcn_update_dpp(x, x, 0x4e, 0xf, 0xf, false);  // quad_perm 2,3,0,1
  if constexpr (M == 4) {
    const int32_t fwd = __builtin_amdgcn_update_dpp(x, x, 0x104, 0xf, 0xf, false);      // row_shl:4
    const int32_t bwd = __builtin_amdgcn_update_dpp(x, x, 0x114, 0xf, 0xf, false);      // row_shr:4
    return (lane & 4) ? bwd : fwd;
  }
  if constexpr (M == 8) return __builtin_amdgcn_update_dpp(x, x, 0x128, 0xf, 0xf, false); // row_ror:8
  return __shfl_xor(x, M);
}

// Inclusive prefix sum over the lanes of a wave: shifted DPP adds within each row, then the
// totals of the rows below added from scalar reads of their last lanes.
__device__ __forceinline__ int32_t wave_incl_sum(int32_t v, int lane) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);         // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);         // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);         // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);         // row_shr:8
  const int32_t r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31),
                r2 = __builtin_amdgcn_readlane(v, 47);
  const int row = lane >> 4;
  return v + (row > 0 ? r0 : 0) + (row > 1 ? r1 : 0) + (row > 2 ? r2 : 0);
}

// ---------------------------------------------------------------------------------------------
// Block map (psa_build_blockmap).
// ---------------------------------------------------------------------------------------------

// Coordinates of entry i of a block map: a one-dimensional block, or a PSABlock-level group.
template <bool GROUPS>
__device__ __forceinline__ int2 map_coord(const Geometry& g, int32_t i) {
  return GROUPS ? group_coord(g, i) : block_coord(g, i);
}

template <bool GROUPS>
__global__ __launch_bounds__(256) void psa_blockmap_kernel(ParamChunk pc, int32_t head0,
                                                           Geometry g, uint8_t* __restrict__ map) {
  const int32_t hc = blockIdx.y;
  const int64_t pairs = (int64_t)g.nb * g.nb;
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= pairs) return;
  const int32_t qb = (int32_t)(p / g.nb), kb = (int32_t)(p - (int64_t)qb * g.nb);
  const bool keep = tile_keep(pc.m[hc], map_coord<GROUPS>(g, qb), map_coord<GROUPS>(g, kb));
  map[(int64_t)(head0 + hc) * pairs + p] = keep ? 1 : 0;
}

// One workgroup per head: per-row counts and the head total (deterministic, no atomics).
template <bool GROUPS>
__global__ __launch_bounds__(256) void psa_rowcount_kernel(ParamChunk pc, int32_t head0,
                                                           Geometry g,
                                                           int32_t* __restrict__ kept_per_row,
                                                           int64_t* __restrict__ kept_per_head) {
  __shared__ int64_t partial[4];
  const int32_t hc = blockIdx.x, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const psa_stripe_t m = pc.m[hc];
  int64_t total = 0;
  for (int32_t qb = wave; qb < g.nb; qb += 4) {
    const int2 cq = map_coord<GROUPS>(g, qb);
    int cnt = 0;
    for (int32_t kb = lane; kb < g.nb; kb += 64)
      cnt += tile_keep(m, cq, map_coord<GROUPS>(g, kb)) ? 1 : 0;
    cnt = wave_sum(cnt);
    if (lane == 0 && kept_per_row) kept_per_row[(int64_t)(head0 + hc) * g.nb + qb] = cnt;
    total += cnt;
  }
  if (lane == 0) partial[wave] = total;
  __syncthreads();
  if (threadIdx.x == 0 && kept_per_head)
    kept_per_head[head0 + hc] = partial[0] + partial[1] + partial[2] + partial[3];
}

template <bool GROUPS>
static hipError_t launch_map(const ParamChunk& pc, int32_t head0, const Geometry& g,
                             uint8_t* blockmap, int32_t* kept_per_row, int64_t* kept_per_head,
                             hipStream_t stream) {
  if (blockmap) {
    const int64_t pairs = (int64_t)g.nb * g.nb;
    dim3 grid((unsigned)((pairs + 255) / 256), (unsigned)pc.n);
    hipLaunchKernelGGL(psa_blockmap_kernel<GROUPS>, grid, dim3(256), 0, stream, pc, head0, g, blockmap);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (kept_per_row || kept_per_head) {
    hipLaunchKernelGGL(psa_rowcount_kernel<GROUPS>, dim3(pc.n), dim3(256), 0, stream, pc, head0, g,
                       kept_per_row, kept_per_head);
    return hipGetLastError();
  }
  return hipSuccess;
}

hipError_t launch_blockmap(const ParamChunk& pc, int32_t head0, const Geometry& g,
                           uint8_t* blockmap, int32_t* kept_per_row, int64_t* kept_per_head,
                           hipStream_t stream) {
  return launch_map<false>(pc, head0, g, blockmap, kept_per_row, kept_per_head, stream);
}

hipError_t launch_group_blockmap(const ParamChunk& pc, int32_t head0, const Geometry& g,
                                 uint8_t* blockmap, int32_t* kept_per_row, int64_t* kept_per_head,
                                 hipStream_t stream) {
  return launch_map<true>(pc, head0, g, blockmap, kept_per_row, kept_per_head, stream);
}

// ---------------------------------------------------------------------------------------------
// PSABlock-centric layout (psa_to_blocks / psa_from_blocks): one workgroup per (batch*head,
// PSABlock), or per 64 text rows; 16-byte chunks, CPR per row.  The blocked side is written or
// read in order, the original side in runs of bw rows.
// ---------------------------------------------------------------------------------------------

// ---------------------------------------------------------------------------------------------
// L2 distance per (batch, head) (the loss of PSA-Search).
// ---------------------------------------------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Fixed-order sum over a 256-thread workgroup (butterfly in each wave, then the four waves).
__device__ __forceinline__ double block_sum(double x, double* red) {
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  const double t = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return t;
}

__global__ __launch_bounds__(256) void psa_l2_partial_kernel(const uint4* __restrict__ o,
                                                             const uint4* __restrict__ ref,
                                                             int64_t vec_per_bh,
                                                             double* __restrict__ partial) {
  __shared__ double red[4];
  const int64_t per = (vec_per_bh + kL2Chunks - 1) / kL2Chunks;
  const int64_t lo = (int64_t)blockIdx.x * per, hi = min(lo + per, vec_per_bh);
  const uint4* a = o + (int64_t)blockIdx.y * vec_per_bh;
  const uint4* b = ref + (int64_t)blockIdx.y * vec_per_bh;
  float se = 0.0f, sr = 0.0f;
  for (int64_t i = lo + threadIdx.x; i < hi; i += 256) {
    const uint4 x = a[i], y = b[i];
    const uint32_t xs[4] = {x.x, x.y, x.z, x.w}, ys[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const float r0 = bf16_lo(ys[j]), r1 = bf16_hi(ys[j]);
      const float d0 = bf16_lo(xs[j]) - r0, d1 = bf16_hi(xs[j]) - r1;
      se = __builtin_fmaf(d0, d0, __builtin_fmaf(d1, d1, se));
      sr = __builtin_fmaf(r0, r0, __builtin_fmaf(r1, r1, sr));
    }
  }
  const double te = block_sum(se, red), tr = block_sum(sr, red);
  if (threadIdx.x == 0) {
    double* dst = partial + ((int64_t)blockIdx.y * kL2Chunks + blockIdx.x) * 2;
    dst[0] = te;
    dst[1] = tr;
  }
}

__global__ __launch_bounds__(64) void psa_l2_final_kernel(const double* __restrict__ partial,
                                                          double* __restrict__ sq_err,
                                                          double* __restrict__ sq_ref) {
  const double* p = partial + (int64_t)blockIdx.x * kL2Chunks * 2;
  double e = p[2 * threadIdx.x], r = p[2 * threadIdx.x + 1];
  for (int off = 32; off > 0; off >>= 1) {
    e += __shfl_xor(e, off);
    r += __shfl_xor(r, off);
  }
  if (threadIdx.x == 0) {
    sq_err[blockIdx.x] = e;
    if (sq_ref) sq_ref[blockIdx.x] = r;
  }
}

hipError_t launch_l2(const void* o, const void* ref, int32_t n_bh, int64_t elems_per_bh,
                     double* partial, double* sq_err, double* sq_ref, hipStream_t stream) {
  static_assert(kL2Chunks == 64, "the final pass sums one partial per lane of a wave");
  hipLaunchKernelGGL(psa_l2_partial_kernel, dim3(kL2Chunks, (unsigned)n_bh), dim3(256), 0, stream,
                     (const uint4*)o, (const uint4*)ref, elems_per_bh / 8, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(psa_l2_final_kernel, dim3((unsigned)n_bh), dim3(64), 0, stream, partial, sq_err,
                     sq_ref);
  return hipGetLastError();
}

template <bool TO, int CPR>
__global__ __launch_bounds__(256) void psa_layout_kernel(const uint4* __restrict__ src,
                                                         uint4* __restrict__ dst, Geometry g) {
  const int32_t n_p = g.tp * g.hp * g.wp;
  const size_t n_orig = (size_t)g.n_video + g.n_text, n_blkd = (size_t)g.n;
  const uint4* s = src + (size_t)blockIdx.y * (TO ? n_orig : n_blkd) * CPR;
  uint4* d = dst + (size_t)blockIdx.y * (TO ? n_blkd : n_orig) * CPR;
  if ((int32_t)blockIdx.x < n_p) {
    const int32_t pb = blockIdx.x, plane = g.hp * g.wp, area = g.pbh * g.pbw;
    const int32_t vol = g.pbt * area;
    const int32_t tq = pb / plane, r = pb - tq * plane, hq = r / g.wp, wq = r - hq * g.wp;
    const int32_t t0 = tq * g.pbt, h0 = hq * g.pbh, w0 = wq * g.pbw;
    // Four 16-byte chunks per thread and round: every load is issued before the first store.
    for (int32_t e0 = threadIdx.x; e0 < vol * CPR; e0 += 4 * 256) {
      size_t from[4], to[4];
      bool live[4];
      uint4 val[4];
#pragma unroll
      for (int u = 0; u < 4; u++) {
        const int32_t e = e0 + u * 256;
        const int32_t x = e / CPR, c = e % CPR;
        const int32_t it = x / area, r2 = x - it * area, ih = r2 / g.pbw, iw = r2 - ih * g.pbw;
        const int32_t t = t0 + it, h = h0 + ih, w = w0 + iw;
        const bool valid = e < vol * CPR && t < g.frames && h < g.height && w < g.width;
        const size_t orow = ((size_t)t * g.height + h) * g.width + w;
        const size_t brow = (size_t)pb * vol + x;
        from[u] = (TO ? orow : brow) * CPR + c;
        to[u] = (TO ? brow : orow) * CPR + c;
        live[u] = TO ? e < vol * CPR : valid;
        val[u] = valid ? s[from[u]] : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int u = 0; u < 4; u++)
        if (live[u]) d[to[u]] = val[u];
    }
  } else {
    const int32_t r0 = ((int32_t)blockIdx.x - n_p) * 64;
    for (int32_t e = threadIdx.x; e < 64 * CPR; e += 256) {
      const int32_t rr = r0 + e / CPR, c = e % CPR;
      if (rr < g.n_text) {
        const size_t orow = (size_t)g.n_video + rr, brow = (size_t)g.n_blk + rr;
        if (TO)
          d[brow * CPR + c] = s[orow * CPR + c];
        else
          d[orow * CPR + c] = s[brow * CPR + c];
      }
    }
  }
}

template <bool TO, int CPR>
static hipError_t launch_layout_t(const void* src, void* dst, int32_t n_bh, const Geometry& g,
                                  hipStream_t stream) {
  const int32_t n_p = g.tp * g.hp * g.wp;
  dim3 grid((unsigned)(n_p + (g.n_text + 63) / 64), (unsigned)n_bh);
  hipLaunchKernelGGL((psa_layout_kernel<TO, CPR>), grid, dim3(256), 0, stream, (const uint4*)src,
                     (uint4*)dst, g);
  return hipGetLastError();
}

hipError_t launch_layout(const void* src, void* dst, int32_t n_bh, int32_t head_dim,
                         const Geometry& g, bool to_blocks, hipStream_t stream) {
  if (head_dim == 128)
    return to_blocks ? launch_layout_t<true, 16>(src, dst, n_bh, g, stream)
                     : launch_layout_t<false, 16>(src, dst, n_bh, g, stream);
  if (head_dim == 64)
    return to_blocks ? launch_layout_t<true, 8>(src, dst, n_bh, g, stream)
                     : launch_layout_t<false, 8>(src, dst, n_bh, g, stream);
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------------------------
// Scheduler pre-pass (psa_attention_fwd).
// ---------------------------------------------------------------------------------------------

WorkspaceLayout workspace_layout(int32_t batch, int32_t n_heads, int32_t nb, bool masks) {
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t items = (size_t)batch * n_heads * nb;
  WorkspaceLayout wl;
  wl.header = 0;
  wl.params = up(wl.header + sizeof(PlanHeader));
  wl.coords = up(wl.params + sizeof(psa_stripe_t) * (size_t)n_heads);
  wl.counts = up(wl.coords + sizeof(int2) * (size_t)nb);
  wl.order = up(wl.counts + sizeof(int32_t) * items);
  wl.queues = up(wl.order + sizeof(int32_t) * items);
  wl.sigs = up(wl.queues + sizeof(int32_t) * kQueueWords);
  wl.pairs = up(wl.sigs + sizeof(uint64_t) * (size_t)n_heads * nb);
  const size_t pair_items = (size_t)batch * n_heads * pairs_per_head(nb);
  wl.spans = up(wl.pairs + sizeof(int2) * (size_t)n_heads * pairs_per_head(nb));
  wl.runspans = up(wl.spans + sizeof(uint32_t) * pair_items);
  wl.starts = up(wl.runspans + sizeof(uint32_t) * pair_items);
  wl.masks = up(wl.starts + sizeof(int32_t) * pair_items);
  wl.total = masks ? up(wl.masks + 2 * sizeof(uint64_t) * (size_t)nb) : wl.masks;
  return wl;
}

// Copies one chunk of stripe parameters into the workspace; the first chunk also invalidates
// the plan header (write_coords != 0) and writes the block coordinate table of one-dimensional
// blocks (write_coords == 1; 3D tiles get theirs from psa_tiles3d_kernel).
__global__ __launch_bounds__(256) void psa_setup_kernel(ParamChunk pc, int32_t head0, Geometry g,
                                                        PlanHeader* __restrict__ header,
                                                        psa_stripe_t* __restrict__ params,
                                                        int2* __restrict__ coords,
                                                        int32_t write_coords) {
  const int32_t i = blockIdx.x * 256 + threadIdx.x;
  if (write_coords && i == 0) header->magic = 0;
  if (i < pc.n) params[head0 + i] = pc.m[i];
  if (write_coords == 1 && i < g.nb) coords[i] = block_coord(g, i);
}

// One wave per tile of the PSABlock-centric layout: the valid positions of the tile (bit r of
// word r / 64) and its coordinates, kDeadTile when it holds only padding.
__global__ __launch_bounds__(256) void psa_tiles3d_kernel(Geometry g, int2* __restrict__ coords,
                                                          uint64_t* __restrict__ masks) {
  const int32_t b = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (b >= g.nb) return;
  const int32_t i0 = b * g.block;
  const uint64_t lo = __builtin_amdgcn_ballot_w64(lane < g.block && position_valid(g, i0 + lane));
  const uint64_t hi = g.block > 64 ? __builtin_amdgcn_ballot_w64(position_valid(g, i0 + 64 + lane))
                                   : ~0ull;
  if (lane == 0) {
    masks[2 * b] = lo;
    masks[2 * b + 1] = hi;
    const bool dead = lo == 0 && (g.block <= 64 || hi == 0);
    coords[b] = dead ? make_int2(kDeadTile, 0) : tile_coord3d(g, b);
  }
}

hipError_t launch_setup(const ParamChunk& pc, int32_t head0, const Geometry& g, void* workspace,
                        const WorkspaceLayout& wl, bool write_coords, hipStream_t stream) {
  char* ws = (char*)workspace;
  const bool blocks3d = g.pbt > 0;
  const bool coords1d = write_coords && !blocks3d;
  const int32_t n = coords1d ? max(g.nb, pc.n) : pc.n;
  hipLaunchKernelGGL(psa_setup_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, pc, head0, g,
                     (PlanHeader*)(ws + wl.header), (psa_stripe_t*)(ws + wl.params),
                     (int2*)(ws + wl.coords), (int32_t)(write_coords ? (coords1d ? 1 : 2) : 0));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !write_coords || !blocks3d) return e;
  hipLaunchKernelGGL(psa_tiles3d_kernel, dim3((g.nb + 3) / 4), dim3(256), 0, stream, g,
                     (int2*)(ws + wl.coords), (uint64_t*)(ws + wl.masks));
  return hipGetLastError();
}

// A 64-bit mix of a block index (the splitmix64 finalizer); the XOR of the mixes of a kept set
// is a hash of the set that does not depend on the order of its members.
__device__ __forceinline__ uint64_t mix64(uint64_t x) {
  x += 0x9e3779b97f4a7c15ull;
  x = (x ^ (x >> 30)) * 0xbf58476d1ce4e5b9ull;
  x = (x ^ (x >> 27)) * 0x94d049bb133111ebull;
  return x ^ (x >> 31);
}

// One wave per work item (batch, head, query block): number of kept key blocks (counts, or
// nullptr), and for the items of the first batch element the per-row count (kept_per_row) and
// the signature of the kept set (sigs), each if asked.
__global__ __launch_bounds__(256) void psa_count_kernel(const psa_stripe_t* __restrict__ params,
                                                        const int2* __restrict__ coords,
                                                        int32_t* __restrict__ counts,
                                                        int32_t* __restrict__ kept_per_row,
                                                        uint64_t* __restrict__ sigs,
                                                        int32_t n_items, int32_t n_heads,
                                                        int32_t nb) {
  const int32_t item = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (item >= n_items) return;
  const int32_t bh = item / nb, qb = item - bh * nb, h = bh % n_heads;
  const psa_stripe_t m = params[h];
  const int2 cq = coords[qb];
  int cnt = 0;
  uint64_t sig = 0;
  for (int32_t kb = lane; kb < nb; kb += 64) {
    const bool keep = tile_keep(m, cq, coords[kb]);
    cnt += keep ? 1 : 0;
    sig ^= keep ? mix64((uint64_t)kb) : 0ull;
  }
  cnt = wave_sum(cnt);
  for (int off = 32; off > 0; off >>= 1) sig ^= __shfl_xor(sig, off);
  if (lane == 0) {
    if (counts) counts[item] = cnt;
    if (bh < n_heads) {
      if (kept_per_row) kept_per_row[(int64_t)h * nb + qb] = cnt;
      if (sigs) sigs[(int64_t)h * nb + qb] = sig;
    }
  }
}

// Exclusive prefix sum (OP = +) or inclusive running maximum (OP = max) over v[0 .. n) in LDS by
// a 1024-thread workgroup; n <= 8 * 1024.  Returns the total (sum) or the last value (max).
template <bool MAX>
__device__ int32_t block_scan(int32_t* v, int32_t n, int32_t* part) {
  constexpr int E = 8;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int32_t loc[E];
  int32_t acc = MAX ? -1 : 0;
#pragma unroll
  for (int e = 0; e < E; e++) {
    const int32_t i = tid * E + e;
    const int32_t x = i < n ? v[i] : (MAX ? -1 : 0);
    loc[e] = acc;                                         // exclusive within the thread
    acc = MAX ? max(acc, x) : acc + x;
  }
  int32_t incl = acc;                                     // inclusive over the wave
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t t = __shfl_up(incl, off);
    if (lane >= off) incl = MAX ? max(incl, t) : incl + t;
  }
  if (lane == 63) part[wave] = incl;
  __syncthreads();
  int32_t before = MAX ? -1 : 0;                          // over the waves before this one
  for (int w = 0; w < wave; w++) before = MAX ? max(before, part[w]) : before + part[w];
  int32_t total = MAX ? -1 : 0;
  for (int w = 0; w < 16; w++) total = MAX ? max(total, part[w]) : total + part[w];
  const int32_t lane_excl = __shfl_up(incl, 1);
  const int32_t prior = lane == 0 ? before : (MAX ? max(before, lane_excl) : before + lane_excl);
#pragma unroll
  for (int e = 0; e < E; e++) {
    const int32_t i = tid * E + e;
    if (i < n) {
      if (MAX)
        v[i] = max(prior, max(loc[e], v[i]));             // inclusive running maximum
      else
        v[i] = prior + loc[e];
    }
  }
  __syncthreads();
  return total;
}

// One workgroup per head: pairs of query blocks for the pair engine.  The rows are sorted by the
// signature of their kept set (then by index); within a run of equal signatures consecutive
// rows pair up.  The rows left over pair up consecutively in one of two orders, chosen from the
// head's stripes: index order (neighbouring slots of one frame), or slot-major (one slot in
// neighbouring frames) where a one-frame shift widens the kept set less than a one-slot shift.
// A shift by one position grows an axis' kept set by (w + 1) / w for a stripe narrower than its
// stride and leaves a full axis unchanged, so slot-major is taken when the spatial stripes are
// partial and the temporal ones either cover their axis or are wider (T_w > S_w).
// pairs[h][p] = (first row, second row or -1), in the order of the first rows.  Rows with
// equal kept sets share every key block, so most pairs of the stripe patterns waste no work;
// the pairing only affects speed, the run decodes each row's own kept set.
constexpr int kPairSort = 8192;                 // a power of two >= PSA_MAX_BLOCKS
__global__ __launch_bounds__(1024) void psa_pairing_kernel(const uint64_t* __restrict__ sigs,
                                                           const psa_stripe_t* __restrict__ params,
                                                           const int2* __restrict__ coords,
                                                           int2* __restrict__ pairs, int32_t nb) {
  __shared__ uint64_t key[kPairSort];         // sorted (signature, row); later leftover rows
  __shared__ int32_t run[kPairSort];          // start of each sorted position's run
  __shared__ int16_t partner[kPairSort];      // by row: partner (first row), -1 single, -2 second
  __shared__ int32_t part[16];
  const int tid = threadIdx.x, lane = tid & 63;
  const uint64_t* sg = sigs + (size_t)blockIdx.x * nb;
  int32_t n2 = 1;
  while (n2 < nb) n2 <<= 1;
  for (int32_t i = tid; i < n2; i += 1024) {
    key[i] = i < nb ? ((sg[i] >> 13) << 13) | (uint64_t)i : ~0ull;
    partner[i] = -3;
  }
  __syncthreads();
  // Bitonic sort of key[0 .. n2), ascending.  Partners 64 or more apart meet in LDS (one
  // barrier per step); the steps of a stage with partners less than 64 apart run inside each
  // wave, on registers exchanged across lanes, with one barrier for all of them.
  auto sort_keys = [&]() {
    for (int32_t k = 2; k <= n2; k <<= 1) {
      int32_t j = k >> 1;
      for (; j >= 64; j >>= 1) {
        for (int32_t i = tid; i < n2; i += 1024) {
          const int32_t ixj = i ^ j;
          if (ixj > i) {
            const uint64_t a = key[i], b = key[ixj];
            if ((a > b) == ((i & k) == 0)) {
              key[i] = b;
              key[ixj] = a;
            }
          }
        }
        __syncthreads();
      }
      for (int32_t i = tid; i < n2; i += 1024) {        // n2 < 64, or whole waves
        uint64_t x = key[i];
        const bool up = (i & k) == 0;
        auto step = [&](auto m) {
          constexpr int M = decltype(m)::value;
          if (M > j) return;
          const uint64_t y = ((uint64_t)(uint32_t)lane_xor<M>((int32_t)(x >> 32), lane) << 32) |
                             (uint32_t)lane_xor<M>((int32_t)(uint32_t)x, lane);
          x = (((i & M) == 0) == up) ? min(x, y) : max(x, y);
        };
        step(std::integral_constant<int, 32>());
        step(std::integral_constant<int, 16>());
        step(std::integral_constant<int, 8>());
        step(std::integral_constant<int, 4>());
        step(std::integral_constant<int, 2>());
        step(std::integral_constant<int, 1>());
        key[i] = x;
      }
      __syncthreads();
    }
  };
  sort_keys();
  auto row_of = [&](int32_t i) { return (int32_t)(key[i] & 8191u); };
  auto same = [&](int32_t i, int32_t j) { return (key[i] >> 13) == (key[j] >> 13); };
  for (int32_t i = tid; i < nb; i += 1024) run[i] = (i == 0 || !same(i, i - 1)) ? i : -1;
  __syncthreads();
  block_scan<true>(run, nb, part);
  for (int32_t i = tid; i < nb; i += 1024) {
    if (((i - run[i]) & 1) != 0) continue;
    const int32_t r = row_of(i);
    if (i + 1 < nb && run[i + 1] == run[i]) {
      const int32_t r2 = row_of(i + 1);
      partner[min(r, r2)] = (int16_t)max(r, r2);
      partner[max(r, r2)] = -2;
    } else {
      partner[r] = -4;                                  // left over
    }
  }
  __syncthreads();
  // Leftover rows: rank in the chosen order (a prefix sum over the rows gives index order), pair
  // ranks 2k and 2k + 1.
  const psa_stripe_t m = params[blockIdx.x];
  const bool slot_major = m.s_w < m.s_s && (m.t_w >= m.t_s || m.t_w > m.s_w);
  for (int32_t i = tid; i < nb; i += 1024) run[i] = partner[i] == -4 ? 1 : 0;
  __syncthreads();
  const int32_t n_left = block_scan<false>(run, nb, part);
  uint32_t* left = (uint32_t*)key;                        // rank -> row
  if (!slot_major) {
    for (int32_t i = tid; i < nb; i += 1024)
      if (partner[i] == -4) left[run[i]] = (uint32_t)i;
  } else {
    // Sort the leftover rows by (slot, frame, row); other rows sort last.  Coordinates beyond
    // the fields (global and padding blocks have negative frames) are clamped: any order is a
    // valid pairing.
    for (int32_t i = tid; i < n2; i += 1024) {
      uint64_t kk = ~0ull;
      if (i < nb && partner[i] == -4) {
        const int2 c = coords[i];
        kk = ((uint64_t)min((uint32_t)c.y, (1u << 26) - 1) << 38) |
             ((uint64_t)min((uint32_t)c.x, (1u << 25) - 1) << 13) | (uint64_t)i;
      }
      key[i] = kk;
    }
    __syncthreads();
    sort_keys();
    // left[] overlays key[]: every thread reads its sorted rows before any is written.
    uint32_t rows[kPairSort / 1024];
#pragma unroll
    for (int j = 0; j < kPairSort / 1024; j++) {
      const int32_t r = tid + 1024 * j;
      rows[j] = r < n_left ? (uint32_t)(key[r] & 8191u) : 0u;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kPairSort / 1024; j++) {
      const int32_t r = tid + 1024 * j;
      if (r < n_left) left[r] = rows[j];
    }
    __syncthreads();
    for (int32_t r = tid; r < n_left; r += 1024) run[left[r]] = r;
  }
  __syncthreads();
  for (int32_t i = tid; i < nb; i += 1024)
    if (partner[i] == -4) {
      const int32_t r = run[i];
      partner[i] = (r & 1) ? -2 : (r + 1 < n_left ? (int16_t)left[r + 1] : -1);
    }
  __syncthreads();
  // Pairs in the order of their first rows.
  for (int32_t i = tid; i < nb; i += 1024) run[i] = partner[i] >= -1 ? 1 : 0;
  __syncthreads();
  block_scan<false>(run, nb, part);
  int2* dst = pairs + (size_t)blockIdx.x * pairs_per_head(nb);
  for (int32_t i = tid; i < nb; i += 1024)
    if (partner[i] >= -1 && run[i] < pairs_per_head(nb)) dst[run[i]] = make_int2(i, partner[i]);
}

// One wave per pair item (batch, head, pair): number of key blocks kept by either row, and the
// first and last of them that are not global (video blocks; the span the start of the item's
// stream is placed in).
__global__ __launch_bounds__(256) void psa_paircount_kernel(const psa_stripe_t* __restrict__ params,
                                                            const int2* __restrict__ coords,
                                                            const int2* __restrict__ pairs,
                                                            int32_t* __restrict__ counts,
                                                            uint32_t* __restrict__ spans,
                                                            int32_t n_items, int32_t n_heads,
                                                            int32_t nb) {
  const int32_t np = pairs_per_head(nb);
  const int32_t item = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (item >= n_items) return;
  const int32_t bh = item / np, p = item - bh * np, h = bh % n_heads;
  const psa_stripe_t m = params[h];
  const int2 pr = pairs[(int64_t)h * np + p];
  const int2 ca = coords[pr.x];
  const int2 cb = pr.y >= 0 ? coords[pr.y] : make_int2(kDeadTile, 0);
  int cnt = 0, lo = nb, hi = -1;
  for (int32_t kb = lane; kb < nb; kb += 64) {
    const int2 ck = coords[kb];
    const bool keep = tile_keep(m, ca, ck) || tile_keep(m, cb, ck);
    cnt += keep ? 1 : 0;
    if (keep && ck.x >= 0) {
      lo = min(lo, kb);
      hi = max(hi, kb);
    }
  }
  cnt = wave_sum(cnt);
  for (int off = 32; off > 0; off >>= 1) {
    lo = min(lo, __shfl_xor(lo, off));
    hi = max(hi, __shfl_xor(hi, off));
  }
  if (lane == 0) {
    counts[item] = cnt;
    spans[item] = hi < 0 ? 0xffffffffu : ((uint32_t)lo | ((uint32_t)hi << 16));
  }
}

// Work estimate of an item, in tiles: kept key blocks plus a fixed cost for loading Q,
// decoding the list and the epilogue.
constexpr int kItemOverhead = 2;

// An item whose work exceeds kLongFactor times the mean item work is scheduled ahead of all
// others (for example the rows of the global text tokens, which keep every key block): taken
// late, one such item would still run long after the rest of the device has drained.
constexpr int kLongFactor = 3;
// Long items are sorted into this many classes of equal width in [0, max work].
constexpr int kWorkClasses = 64;
constexpr int kScheduleWaves = 16;

// Single workgroup.  Every queue x (the XCD of the workgroups that start on it) begins with its
// share of the long items, longest first and dealt round-robin over the queues.  The other items
// follow head by head: the (batch, head) pairs are ordered by their work, longest first, and
// every head's query blocks are cut into kNumQueues contiguous ranges of equal work, queue x
// listing range x of every head.  All XCDs therefore sweep the heads together -- the K/V of the
// one or two heads in flight stay in the memory-side cache -- and the workgroups of one XCD
// stream neighbouring key blocks through its L2.
__global__ __launch_bounds__(1024) void psa_schedule_kernel(const int32_t* __restrict__ counts,
                                                            int32_t* __restrict__ order,
                                                            int32_t* __restrict__ queues,
                                                            PlanHeader* __restrict__ header,
                                                            PlanHeader done, int32_t nb,
                                                            int32_t write_header,
                                                            const uint32_t* __restrict__ spans,
                                                            uint32_t* __restrict__ runspans) {
  const int32_t n_bh = done.n_bh, n = n_bh * nb;
  __shared__ int64_t total[PSA_MAX_BATCH_HEADS];
  __shared__ int32_t by_rank[PSA_MAX_BATCH_HEADS];
  __shared__ uint16_t bounds[PSA_MAX_BATCH_HEADS][kNumQueues + 1];
  __shared__ int32_t qoff[PSA_MAX_BATCH_HEADS][kNumQueues];
  __shared__ int32_t hist[kScheduleWaves][kWorkClasses];
  __shared__ int32_t qstart[kNumQueues + 1];
  __shared__ uint64_t all_work;
  __shared__ int32_t max_count, n_long;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;

  if (tid == 0) {
    all_work = 0;
    max_count = 0;
  }
  for (int32_t i = tid; i < kScheduleWaves * kWorkClasses; i += 1024) (&hist[0][0])[i] = 0;
  __syncthreads();
  constexpr int kLoads = 4;                 // loads in flight per lane in the sweeps below
  // Sums of one pair's work stay below 2^31: at most PSA_MAX_BLOCKS items of at most
  // PSA_MAX_BLOCKS + kItemOverhead tiles.
  for (int32_t bh = wave; bh < n_bh; bh += kScheduleWaves) {
    int32_t s = 0;
    int32_t mx = 0;
    for (int32_t q0 = lane; q0 < nb; q0 += 64 * kLoads) {
      int32_t c[kLoads];
#pragma unroll
      for (int j = 0; j < kLoads; j++) c[j] = q0 + 64 * j < nb ? counts[bh * nb + q0 + 64 * j] : -1;
#pragma unroll
      for (int j = 0; j < kLoads; j++) {
        s += c[j] < 0 ? 0 : c[j] + kItemOverhead;
        mx = max(mx, c[j]);
      }
    }
    s = wave_reduce<0>(s);
    mx = wave_reduce<2>(mx);
    if (lane == 0) {
      total[bh] = s;
      atomicAdd(&all_work, (uint64_t)s);
      atomicMax(&max_count, mx);
    }
  }
  __syncthreads();
  const int64_t long_above = (int64_t)kLongFactor * (int64_t)all_work;
  auto work_of = [&](int32_t item) { return (int64_t)counts[item] + kItemOverhead; };
  // Whether any item is long follows from the largest one; without long items every pass that
  // looks for them is skipped.
  const bool any_long = ((int64_t)max_count + kItemOverhead) * n > long_above;
  auto is_long = [&](int32_t item) { return any_long && work_of(item) * n > long_above; };
  if (any_long) {
    // Work of each pair without its long items.
    for (int32_t bh = wave; bh < n_bh; bh += kScheduleWaves) {
      int32_t s = 0;
      for (int32_t q0 = lane; q0 < nb; q0 += 64 * kLoads) {
        int64_t w[kLoads];
#pragma unroll
        for (int j = 0; j < kLoads; j++) w[j] = q0 + 64 * j < nb ? work_of(bh * nb + q0 + 64 * j) : 0;
#pragma unroll
        for (int j = 0; j < kLoads; j++) s += w[j] * n > long_above ? 0 : (int32_t)w[j];
      }
      s = wave_reduce<0>(s);
      if (lane == 0) total[bh] = s;
    }
    __syncthreads();
  }
  for (int32_t bh = tid; bh < n_bh; bh += 1024) {
    int32_t r = 0;
    const int64_t mine = total[bh];
    for (int32_t j = 0; j < n_bh; j++) r += (total[j] > mine || (total[j] == mine && j < bh)) ? 1 : 0;
    by_rank[r] = bh;
  }
  __syncthreads();

  // Equal-work ranges of each head over its other items: bounds[r][x] = first query block of
  // range x.
  for (int32_t r = wave; r < n_bh; r += kScheduleWaves) {
    const int32_t bh = by_rank[r];
    const int64_t head_total = total[bh];
    int32_t base = 0;
    int32_t next = 1;                       // next boundary to place
    if (lane == 0) bounds[r][0] = 0;
    for (int32_t g0 = 0; g0 < nb && next < kNumQueues; g0 += 64 * kLoads) {
      int32_t wv[kLoads];
#pragma unroll
      for (int j = 0; j < kLoads; j++) {
        const int32_t qb = g0 + 64 * j + lane;
        wv[j] = qb < nb && !is_long(bh * nb + qb) ? (int32_t)work_of(bh * nb + qb) : 0;
      }
#pragma unroll
      for (int j = 0; j < kLoads; j++) {
        const int32_t q0 = g0 + 64 * j, qb = q0 + lane;
        const int32_t w = wv[j];
        const int32_t incl = wave_incl_sum(w, lane);        // inclusive prefix over the wave
        const int64_t excl = base + incl - w;
        // range x starts at the first block whose preceding work reaches x/Q of the head
        while (next < kNumQueues) {
          const int64_t target = head_total * next / kNumQueues;
          const uint64_t hit = __builtin_amdgcn_ballot_w64(qb < nb && excl >= target);
          if (!hit) break;
          const int32_t first = q0 + __builtin_ctzll(hit);
          if (lane == 0) bounds[r][next] = (uint16_t)first;
          next++;
        }
        base += __builtin_amdgcn_readlane(incl, 63);
      }
    }
    for (; next < kNumQueues; next++)
      if (lane == 0) bounds[r][next] = (uint16_t)nb;
    if (lane == 0) bounds[r][kNumQueues] = (uint16_t)nb;
  }

  // Long items: stable class sort.  Entry s of the unsorted list is query block s mod nb of the
  // pair of rank s div nb; wave w owns the slice [w n / W, (w + 1) n / W).  Class 0 holds the
  // longest items.
  const int32_t lo = (int32_t)((int64_t)n * wave / kScheduleWaves);
  const int32_t hi = (int32_t)((int64_t)n * (wave + 1) / kScheduleWaves);
  const int32_t top = max_count + 1;
  auto item_of = [&](int32_t s) { const int32_t r = s / nb; return by_rank[r] * nb + (s - r * nb); };
  auto class_of = [&](int32_t item) {
    return kWorkClasses - 1 - (int32_t)((int64_t)counts[item] * kWorkClasses / top);
  };
  if (any_long)
    for (int32_t s = lo + lane; s < hi; s += 64) {
      const int32_t item = item_of(s);
      if (is_long(item)) atomicAdd(&hist[wave][class_of(item)], 1);
    }
  __syncthreads();

  // Number of the other items in every (head, queue) range, one wave per range.
  for (int32_t pair = wave; pair < n_bh * kNumQueues; pair += kScheduleWaves) {
    const int32_t r = pair / kNumQueues, x = pair - r * kNumQueues;
    const int32_t item0 = by_rank[r] * nb, end = bounds[r][x + 1];
    int32_t c = end - bounds[r][x];
    if (any_long)
      for (int32_t qb = bounds[r][x] + lane; __builtin_amdgcn_readfirstlane(qb - lane) < end; qb += 64)
        c -= __builtin_popcountll(__builtin_amdgcn_ballot_w64(qb < end && is_long(item0 + qb)));
    if (lane == 0) qoff[r][x] = c;
  }
  // Exclusive scan of the class histogram in (class, wave) order: hist[w][c] becomes the first
  // list position of the class-c long items of slice w.
  if (wave == 0) {
    int32_t col = 0;
    for (int w = 0; w < kScheduleWaves; w++) col += hist[w][lane];
    int32_t incl = col;
    for (int off = 1; off < 64; off <<= 1) {
      const int32_t t = __shfl_up(incl, off);
      if (lane >= off) incl += t;
    }
    int32_t pos = incl - col;
    for (int w = 0; w < kScheduleWaves; w++) {
      const int32_t h = hist[w][lane];
      hist[w][lane] = pos;
      pos += h;
    }
    if (lane == 63) n_long = incl;
  }
  __syncthreads();
  // Offsets of each head's range inside its queue, and the queue starts: queue x holds long
  // list positions x, x + Q, ... (n_long div Q of them, one more for x < n_long mod Q), then
  // its ranges.
  if (tid < kNumQueues) {
    int32_t acc = n_long / kNumQueues + (tid < n_long % kNumQueues ? 1 : 0);
    for (int32_t r = 0; r < n_bh; r++) {
      const int32_t c = qoff[r][tid];
      qoff[r][tid] = acc;
      acc += c;
    }
    qstart[tid + 1] = acc;                  // length, turned into a start below
  }
  __syncthreads();
  if (tid == 0) {
    qstart[0] = 0;
    for (int x = 0; x < kNumQueues; x++) qstart[x + 1] += qstart[x];
  }
  __syncthreads();

  // Stable scatter of the long items: the lanes of one 64-entry chunk that share a class are
  // found with one ballot per class bit; each takes the next position of its class in the order
  // of its lane.
  for (int32_t s0 = lo; any_long && s0 < hi; s0 += 64) {
    const int32_t s = s0 + lane;
    const int32_t item = s < hi ? item_of(s) : 0;
    const bool valid = s < hi && is_long(item);
    if (!__builtin_amdgcn_ballot_w64(valid)) continue;
    const int32_t cls = valid ? class_of(item) : 0;
    uint64_t same = __builtin_amdgcn_ballot_w64(valid);
    for (int bit = 1; bit < kWorkClasses; bit <<= 1) {
      const uint64_t ones = __builtin_amdgcn_ballot_w64(valid && (cls & bit));
      same &= (cls & bit) ? ones : ~ones;
    }
    const int32_t base = valid ? hist[wave][cls] : 0;
    __builtin_amdgcn_wave_barrier();
    if (valid) {
      const int32_t pos = base + __builtin_popcountll(same & ((1ull << lane) - 1));
      order[qstart[pos % kNumQueues] + pos / kNumQueues] = item;
      if (runspans) runspans[item] = spans[item];        // a long item is a run of its own
      if (__builtin_ctzll(same) == lane) hist[wave][cls] = base + __builtin_popcountll(same);
    }
    __builtin_amdgcn_wave_barrier();
  }
  // Each wave takes ranges W, W + 16, ...; the count and span of the first 64 items of the next
  // range are loaded while the current one is written.
  const int32_t n_ranges = n_bh * kNumQueues;
  auto head_of = [&](int32_t range, int32_t& cnt, uint32_t& span) {
    cnt = 0;
    span = 0xffffffffu;
    if (range >= n_ranges) return;
    const int32_t r = range / kNumQueues, x = range - r * kNumQueues;
    const int32_t qb = bounds[r][x] + lane;
    if (qb >= bounds[r][x + 1]) return;
    if (any_long) cnt = counts[by_rank[r] * nb + qb];
    if (runspans) span = spans[by_rank[r] * nb + qb];
  };
  int32_t next_cnt;
  uint32_t next_span;
  head_of(wave, next_cnt, next_span);
  for (int32_t range = wave; range < n_ranges; range += kScheduleWaves) {
    const int32_t head_cnt = next_cnt;
    const uint32_t head_span = next_span;
    head_of(range + kScheduleWaves, next_cnt, next_span);
    const int32_t r = range / kNumQueues, x = range - r * kNumQueues;
    const int32_t item0 = by_rank[r] * nb, begin = bounds[r][x], end = bounds[r][x + 1];
    int32_t* dst = order + qstart[x] + qoff[r][x];
    int32_t lo = 0xffff, hi = 0;
    bool head_keep = false;
    for (int32_t qb = begin + lane; __builtin_amdgcn_readfirstlane(qb - lane) < end; qb += 64) {
      const bool head = qb - lane == begin;
      const int32_t cnt = head ? head_cnt : (any_long && qb < end ? counts[item0 + qb] : 0);
      const uint32_t span = head ? head_span : (runspans && qb < end ? spans[item0 + qb] : 0xffffffffu);
      const bool keep = qb < end && !(any_long && ((int64_t)cnt + kItemOverhead) * n > long_above);
      if (head) head_keep = keep;
      const uint64_t mask = __builtin_amdgcn_ballot_w64(keep);
      if (keep) dst[__builtin_popcountll(mask & ((1ull << lane) - 1))] = item0 + qb;
      dst += __builtin_popcountll(mask);
      if (keep && span != 0xffffffffu) {
        lo = min(lo, (int32_t)(span & 0xffffu));
        hi = max(hi, (int32_t)(span >> 16));
      }
    }
    if (runspans) {
      // the run's span: the union of its items' spans of non-global blocks
      lo = wave_reduce<1>(lo);
      hi = wave_reduce<2>(hi);
      const uint32_t run = lo > hi ? 0xffffffffu : ((uint32_t)lo | ((uint32_t)hi << 16));
      for (int32_t qb = begin + lane; qb < end; qb += 64)
        if (qb - lane == begin ? head_keep : !is_long(item0 + qb)) runspans[item0 + qb] = run;
    }
  }
  if (tid <= kNumQueues) queues[tid] = qstart[tid];
  if (tid < kNumQueues) queues[kQueueCounters + tid * kCounterStride] = 0;
  if (tid == 0) queues[kStartsDone] = 0;
  __syncthreads();
  if (tid == 0 && write_header) {
    __threadfence();
    *header = done;
  }
}

// Where each pair item's K/V stream starts.  The workgroups of one XCD share its L2, and a K/V
// block stays there for only about two block steps of the XCD's 32 workgroups; so a block is
// reused only when the items in flight on the XCD read it at nearly the same time.  Each item
// therefore starts its cyclic walk over its key blocks where the item started just before it on
// the same queue is predicted to be by then: the queue is replayed with 32 workgroups taking
// items as they become free (work = kept blocks + item overhead, the schedule's estimate), and
// the predecessor's position is placed by linear interpolation over the span of non-global key
// blocks of their run.  Items that keep every key block start at block 0 (ascending, as in the
// dense kernel).  The result depends on the plan only, so runs stay deterministic.
// One 1024-thread workgroup per queue, over tiles of kStartsTile queue entries; the last
// workgroup to finish writes the plan header.
//  0. All waves load the tile's items, kept counts and spans into LDS.
//  1. Start times (wave 0): the 32 times at which the XCD's workgroups become free are kept
//     sorted over lanes 0..31; the queue's items are replayed 16 at a time -- they start at the
//     16 earliest free times (this differs from taking them one by one only when an item of the
//     group would end before a later one of the group starts), their workgroups' next free times
//     replace those lanes, and a bitonic sort over the 32 lanes restores the order.
//  2. Start blocks (all waves): within a run (the items of one head's range in the queue), each
//     item starts where its predecessor is predicted to be by then: the predecessor's start block
//     advanced by (its elapsed time / its work) of the run's span, cyclically; a run's first item
//     starts at its own first non-global block.  These are segmented prefix sums: a plain prefix
//     sum over the tile less its value where the item's run began (a running maximum of the run
//     starts), the last item's sum carried into the next tile.
constexpr int kStartGroup = 16;
constexpr uint32_t kNoSpan = 0xffffffffu;

template <int K, int H>
__device__ __forceinline__ int32_t bitonic_step(int32_t v, int lane) {
  const int32_t other = lane_xor<H>(v, lane);
  const bool up = ((lane & K) == 0) == ((lane & H) == 0);
  return up ? min(v, other) : max(v, other);
}

constexpr int kStartsTile = 2048;
static_assert(kStartsTile % kStartGroup == 0, "the replay's groups of a queue must not straddle tiles");
__global__ __launch_bounds__(1024) void psa_starts_kernel(
    const int32_t* __restrict__ counts, const uint32_t* __restrict__ spans,
    const uint32_t* __restrict__ runspans, const int32_t* __restrict__ order,
    int32_t* __restrict__ queues, int32_t* __restrict__ starts, PlanHeader* __restrict__ header,
    PlanHeader done, int32_t np, int32_t nb) {
  constexpr int kSlots = 32;                       // workgroups of one XCD
  constexpr int kPer = kStartsTile / 1024;         // entries per thread in the loads
  __shared__ int32_t s_item[kStartsTile], s_cnt[kStartsTile], s_t[kStartsTile];
  __shared__ uint32_t s_own[kStartsTile], s_run[kStartsTile];
  __shared__ int32_t s_v[kStartsTile], s_sum[kStartsTile], s_seg[kStartsTile];
  __shared__ int32_t part[16];
  __shared__ int32_t c_bh, c_t, c_work, c_acc;     // the entry before the tile
  __shared__ uint32_t c_run;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, queue = blockIdx.x;
  const int32_t q0 = queues[queue], q1 = queues[queue + 1];
  if (tid == 0) {
    c_bh = -1;
    c_t = 0;
    c_work = 1;
    c_acc = 0;
    c_run = kNoSpan;
  }
  int32_t free_at = lane < kSlots ? 0 : INT32_MAX; // wave 0, carried over the tiles
  for (int32_t t0 = q0; t0 < q1; t0 += kStartsTile) {
    const int32_t tn = min(kStartsTile, q1 - t0);
    // 0. loads: every thread issues its item indices, then their counts and spans
    int32_t it[kPer];
#pragma unroll
    for (int r = 0; r < kPer; r++) {
      const int32_t i = tid + 1024 * r;
      it[r] = i < tn ? order[t0 + i] : 0;
    }
#pragma unroll
    for (int r = 0; r < kPer; r++) {
      const int32_t i = tid + 1024 * r;
      if (i < tn) {
        s_item[i] = it[r];
        s_cnt[i] = counts[it[r]];
        s_own[i] = spans[it[r]];
        s_run[i] = runspans[it[r]];
      }
    }
    __syncthreads();
    // 1. start times
    if (wave == 0) {
      int32_t w_next = lane < kStartGroup && lane < tn ? s_cnt[lane] : 0;
      for (int32_t g = 0; g < tn; g += kStartGroup) {
        const int32_t gn = min(kStartGroup, tn - g);
        const int32_t w = w_next;
        w_next = lane < kStartGroup && g + kStartGroup + lane < tn ? s_cnt[g + kStartGroup + lane] : 0;
        if (lane < gn) s_t[g + lane] = free_at;    // lane i: the i-th earliest free time
        free_at += lane < gn ? w + kItemOverhead : 0;
        free_at = bitonic_step<2, 1>(free_at, lane);
        free_at = bitonic_step<4, 2>(free_at, lane);
        free_at = bitonic_step<4, 1>(free_at, lane);
        free_at = bitonic_step<8, 4>(free_at, lane);
        free_at = bitonic_step<8, 2>(free_at, lane);
        free_at = bitonic_step<8, 1>(free_at, lane);
        free_at = bitonic_step<16, 8>(free_at, lane);
        free_at = bitonic_step<16, 4>(free_at, lane);
        free_at = bitonic_step<16, 2>(free_at, lane);
        free_at = bitonic_step<16, 1>(free_at, lane);
        free_at = bitonic_step<32, 16>(free_at, lane);
        free_at = bitonic_step<32, 8>(free_at, lane);
        free_at = bitonic_step<32, 4>(free_at, lane);
        free_at = bitonic_step<32, 2>(free_at, lane);
        free_at = bitonic_step<32, 1>(free_at, lane);
        free_at = lane < kSlots ? free_at : INT32_MAX;
      }
    }
    __syncthreads();
    // 2. each entry's step from its predecessor (v), and where its run began (seg)
    for (int32_t i = tid; i < tn; i += 1024) {
      const int32_t bh = s_item[i] / np, t = s_t[i];
      const uint32_t run = s_run[i], own = s_own[i];
      int32_t p_bh, p_t, p_work;
      uint32_t p_run;
      if (i > 0) {
        p_bh = s_item[i - 1] / np;
        p_t = s_t[i - 1];
        p_work = s_cnt[i - 1] + kItemOverhead;
        p_run = s_run[i - 1];
      } else {
        p_bh = c_bh;
        p_t = c_t;
        p_work = c_work;
        p_run = c_run;
      }
      const bool first = p_bh != bh || p_run != run || t0 + i == q0;
      const int32_t lo = (int32_t)(run & 0xffffu), len = (int32_t)(run >> 16) - lo + 1;
      int32_t v = 0;
      if (run != kNoSpan) {
        if (first)
          v = own != kNoSpan ? (int32_t)(own & 0xffffu) - lo : 0;
        else
          v = min(max(t - p_t, 0), p_work - 1) * len / p_work;   // < 2^13 * 2^13
      }
      s_v[i] = v;
      s_sum[i] = v;
      s_seg[i] = first ? i : -1;
    }
    __syncthreads();
    const int32_t carry = c_acc;
    block_scan<false>(s_sum, tn, part);              // exclusive sums
    block_scan<true>(s_seg, tn, part);               // start of each entry's run, -1: before the tile
    for (int32_t i = tid; i < tn; i += 1024) {
      const int32_t seg = s_seg[i];
      const int32_t acc = s_sum[i] + s_v[i] - (seg >= 0 ? s_sum[seg] : -carry);
      const uint32_t run = s_run[i];
      const int32_t lo = (int32_t)(run & 0xffffu), len = (int32_t)(run >> 16) - lo + 1;
      int32_t kb = run == kNoSpan ? 0 : lo + acc % len;
      if (s_cnt[i] >= nb) kb = 0;
      starts[s_item[i]] = kb;
      if (i == tn - 1) {                             // carry into the next tile
        c_bh = s_item[i] / np;
        c_t = s_t[i];
        c_work = s_cnt[i] + kItemOverhead;
        c_run = run;
        c_acc = acc;
      }
    }
    __syncthreads();
  }
  if (tid == 0) {
    __threadfence();
    if (atomicAdd(&queues[kStartsDone], 1) == kNumQueues - 1) {
      __threadfence();
      *header = done;
    }
  }
}

static PlanHeader plan_header(const Geometry& g, int32_t batch, int32_t n_heads) {
  PlanHeader h;
  h.magic = kPlanMagic;
  h.n_bh = batch * n_heads;
  h.n_heads = n_heads;
  h.nb = g.nb;
  h.block = g.block;
  h.n = g.n;
  h.frames = g.frames;
  h.height = g.height;
  h.width = g.width;
  h.n_text = g.n_text;
  h.pbt = g.pbt;
  h.pbh = g.pbh;
  h.pbw = g.pbw;
  return h;
}

// Whether the attention of this geometry runs on the pair engine (work items are pairs of
// query blocks) or on one query block per work item.
static bool pair_engine(const Geometry& g) { return g.block == 128; }

hipError_t launch_schedule(const Geometry& g, int32_t batch, int32_t n_heads, void* workspace,
                           const WorkspaceLayout& wl, int32_t* kept_per_row, hipStream_t stream) {
  char* ws = (char*)workspace;
  const psa_stripe_t* params = (const psa_stripe_t*)(ws + wl.params);
  const int2* coords = (const int2*)(ws + wl.coords);
  int32_t* counts = (int32_t*)(ws + wl.counts);
  int32_t per_head = g.nb;
  hipError_t e;
  if (pair_engine(g)) {
    // Row counts and kept-set signatures of one batch element, the pairs of each head, then the
    // work of every pair item.
    const int32_t n_rows = n_heads * g.nb;
    hipLaunchKernelGGL(psa_count_kernel, dim3((n_rows + 3) / 4), dim3(256), 0, stream, params, coords,
                       nullptr, kept_per_row, (uint64_t*)(ws + wl.sigs), n_rows, n_heads, g.nb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(psa_pairing_kernel, dim3(n_heads), dim3(1024), 0, stream,
                       (const uint64_t*)(ws + wl.sigs), params, coords, (int2*)(ws + wl.pairs), g.nb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    per_head = pairs_per_head(g.nb);
    const int32_t n_items = batch * n_heads * per_head;
    hipLaunchKernelGGL(psa_paircount_kernel, dim3((n_items + 3) / 4), dim3(256), 0, stream, params, coords,
                       (const int2*)(ws + wl.pairs), counts, (uint32_t*)(ws + wl.spans), n_items, n_heads,
                       g.nb);
  } else {
    const int32_t n_items = batch * n_heads * g.nb;
    hipLaunchKernelGGL(psa_count_kernel, dim3((n_items + 3) / 4), dim3(256), 0, stream, params, coords,
                       counts, kept_per_row, nullptr, n_items, n_heads, g.nb);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(psa_schedule_kernel, dim3(1), dim3(1024), 0, stream, (const int32_t*)counts,
                     (int32_t*)(ws + wl.order), (int32_t*)(ws + wl.queues), (PlanHeader*)(ws + wl.header),
                     plan_header(g, batch, n_heads), per_head, (int32_t)!pair_engine(g),
                     pair_engine(g) ? (const uint32_t*)(ws + wl.spans) : nullptr,
                     pair_engine(g) ? (uint32_t*)(ws + wl.runspans) : nullptr);
  if ((e = hipGetLastError()) != hipSuccess || !pair_engine(g)) return e;
  hipLaunchKernelGGL(psa_starts_kernel, dim3(kNumQueues), dim3(1024), 0, stream, (const int32_t*)counts,
                     (const uint32_t*)(ws + wl.spans), (const uint32_t*)(ws + wl.runspans),
                     (const int32_t*)(ws + wl.order), (int32_t*)(ws + wl.queues), (int32_t*)(ws + wl.starts),
                     (PlanHeader*)(ws + wl.header), plan_header(g, batch, n_heads), per_head, g.nb);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------------
// Tile engine.
// ---------------------------------------------------------------------------------------------

template <int D, int BLK>
struct Tile {
  static constexpr int kWaves = BLK / 32;      // one wave per 32 query rows
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int KT = BLK / 32;          // 32-key row groups of S^T
  static constexpr int DC = D / 16;            // 16-wide head-dim chunks (Q K^T contraction)
  static constexpr int DT = D / 32;            // 32-row head-dim groups of O^T
  static constexpr int KC = BLK / 16;          // 16-key chunks (P V contraction)
  static constexpr int RB = D * 2;             // LDS bytes per row
  static constexpr int CPR = D / 8;            // 16-byte chunks per row
  static constexpr int BYTES = BLK * RB;       // one K or V block in LDS
  static constexpr int LPW = BYTES / (1024 * kWaves);  // 1 KB DMA slots per wave per tensor
  static_assert(LPW >= 1 && BYTES % (1024 * kWaves) == 0, "tile shape");
};

// XOR swizzle of the 16-byte chunks of LDS row `row` (D = 128: 16 chunks per row).  K reads
// touch the 16 rows {x..x+15} (8 lanes per cycle: rows {x..x+3, x+8..x+11}) at one logical
// chunk; transposed V reads touch 4 consecutive rows r0..r0+3 at 4 consecutive chunks (16 lanes
// per cycle: 2 chunks).  Within a quad of rows, bits (1,2) and bits (2,3) of the swizzle are
// both all distinct; row bits 2 and 3 flip bits 1 and 0.  Every one of these access groups then
// hits distinct banks whether the LDS serves 128 or 256 bytes per clock.
template <int CPR>
__device__ __forceinline__ int swz(int row) {
  const int i = row & 3;
  const int s = (((i >> 1) << 3) | ((i & 1) << 2) | ((i >> 1) << 1)) ^ (((row >> 2) & 1) << 1) ^
                ((row >> 3) & 1);
  return s & (CPR - 1);
}

// Lane l supplies K row sigma(l & 31) of a 32-row group so that accumulator element i of lane l
// holds key 16*(i/8) + 8*(l/32) + (i%8).
__device__ __forceinline__ int key_perm(int r) {
  const int a = r >> 3, hh = (r >> 2) & 1, b = r & 3;
  return 16 * (a >> 1) + 8 * hh + 4 * (a & 1) + b;
}

__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}


// Direct global->LDS loads of one half (BLK/2 rows) of a K or V block.  DMA slot j (1 KB) of
// the block covers LDS bytes [1024 j, +1024); lane l writes bytes [1024 j + 16 l, +16): row
// (64 j + l) / CPR, physical chunk (64 j + l) % CPR, which holds logical chunk (physical ^
// swz(row)).  The first half of the slots holds rows 0 .. BLK/2-1.  Every wave loads HW = LPW/2
// slots of each half: slot h*S2 + wave*HW + i for half h, so that each wave issues the same
// number of loads per half.  The loads are issued from inline assembly (SGPR base + 32-bit lane
// offset, M0 = LDS destination); the compiler does not track them, so every consumer first
// waits with wait_dma<N>() and a barrier.
template <int D, int BLK>
struct DmaPlan {
  using T = Tile<D, BLK>;
  static constexpr int HW = T::LPW / 2;                 // slots per wave per half
  static constexpr int S2 = T::LPW * T::kWaves / 2;     // slots per half
  static_assert(T::LPW % 2 == 0, "each wave loads whole slots of both halves");
  uint32_t off[T::LPW];  // byte offset in the block of the 16 bytes this lane loads: [half][i]
  uint32_t lds_k[2];     // LDS byte address of this wave's first slot of each K half
  uint32_t lds_v[2];     // same in the V buffer
  int wave, lane;

  __device__ __forceinline__ void init(uint32_t k_base, uint32_t v_base, int wave_, int lane_) {
    wave = wave_;
    lane = lane_;
#pragma unroll
    for (int i = 0; i < T::LPW; i++) off[i] = offset(i, BLK);
#pragma unroll
    for (int h = 0; h < 2; h++) {
      lds_k[h] = k_base + (uint32_t)(h * S2 + wave * HW) * 1024u;
      lds_v[h] = v_base + (uint32_t)(h * S2 + wave * HW) * 1024u;
    }
  }

  // Offset of entry idx = half * HW + i, with rows at or past `rows` clamped to row rows - 1.
  __device__ __forceinline__ uint32_t offset(int idx, int rows) const {
    const int slot = (idx / HW) * S2 + wave * HW + idx % HW;
    const int p = slot * 64 + lane;
    const int row = p / T::CPR;
    const int chunk = (p % T::CPR) ^ swz<T::CPR>(row);
    return (uint32_t)(min(row, rows - 1) * T::RB + chunk * 16);
  }
};

__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return (uint32_t)(uintptr_t)(const PSA_LDS void*)p;
}

__device__ __forceinline__ void dma16(uint32_t lds_addr, uint32_t voff, const void* base) {
  // One wait state separates the M0 write from the LDS DMA that reads it.
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(lds_addr), "v"(voff), "s"(base)
               : "memory");
}

// Wait until at most N of this wave's DMA loads are outstanding.
template <int N>
__device__ __forceinline__ void wait_dma() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Load half h (rows h*BLK/2 ..) of block kb of one tensor (K or V) into its LDS buffer: this
// wave's HW slots of that half.  Rows past the sequence end are clamped to the last row: their
// scores are masked to -inf, so they are never weighted.
template <int D, int BLK>
__device__ __forceinline__ void issue_half(const DmaPlan<D, BLK>& plan, const __bf16* xh,
                                           const uint32_t (&lds)[2], int h, int kb, int n) {
  using P = DmaPlan<D, BLK>;
  kb = __builtin_amdgcn_readfirstlane(kb);
  const int rows = n - kb * BLK;
  const void* base = (const void*)(xh + (size_t)kb * BLK * D);
  const uint32_t l0 = __builtin_amdgcn_readfirstlane(lds[h]);
  if (rows >= BLK) {
#pragma unroll
    for (int i = 0; i < P::HW; i++) dma16(l0 + i * 1024u, plan.off[h * P::HW + i], base);
  } else {
#pragma unroll
    for (int i = 0; i < P::HW; i++) dma16(l0 + i * 1024u, plan.offset(h * P::HW + i, rows), base);
  }
}

// Per-wave state: 32 query rows (lane l owns row l & 31; lanes l and l^32 split its keys).
// Scores live in the exp2 domain: Q is multiplied by scale*log2(e) once, when it is loaded, and
// the S^T accumulators start at -m instead of 0, so the MFMAs deliver S - m and the softmax needs
// no per-score multiply or subtract.
template <int D, int BLK>
struct WaveState {
  using T = Tile<D, BLK>;
  bf16x8 q[T::DC];     // (scale*log2(e) Q)^T B operands
  f32x16 o[T::DT];     // O^T accumulators
  f32x16 negm;         // -m in all 16 elements (0 while m = -inf): initial S^T accumulator
  float m;             // running max of the scaled scores
  float l;             // running sum of the bf16-rounded P over this lane's keys
};

// Each key/value block is processed in two halves of HK = BLK/2 keys (S^T: HK/32 groups of 32 keys
// per wave); every half updates the online-softmax statistics on its own.
template <int D, int BLK>
struct Half {
  static constexpr int HK = BLK / 2;          // keys per half
  static constexpr int KT = HK / 32;          // 32-key groups of S^T per half
  static constexpr int KC = HK / 16;          // 16-key chunks per half
};

// S^T = K Q^T for keys [k0, k0 + HK) of the block (K rows from LDS).
template <int D, int BLK>
__device__ __forceinline__ void qk_half(const WaveState<D, BLK>& st,
                                        f32x16 (&s)[Half<D, BLK>::KT], const uint8_t* sk, int k0,
                                        int lane) {
  using T = Tile<D, BLK>;
  using H = Half<D, BLK>;
  const int h = lane >> 5;
  const int krow0 = k0 + key_perm(lane & 31);
  const int ksw = swz<T::CPR>(krow0);   // identical for krow0 + 32 kt
  // The K operands of step cc + 1 are read while the MFMAs of step cc run.
  bf16x8 a[2][H::KT];
#pragma unroll
  for (int kt = 0; kt < H::KT; kt++)
    a[0][kt] = *(const bf16x8*)(sk + (krow0 + 32 * kt) * T::RB + ((h ^ ksw) << 4));
#pragma unroll
  for (int cc = 0; cc < T::DC; cc++) {
    if (cc + 1 < T::DC) {
#pragma unroll
      for (int kt = 0; kt < H::KT; kt++)
        a[(cc + 1) & 1][kt] =
            *(const bf16x8*)(sk + (krow0 + 32 * kt) * T::RB + (((2 * (cc + 1) + h) ^ ksw) << 4));
    }
    __builtin_amdgcn_sched_barrier(0);      // keep the reads ahead of this step's MFMAs
#pragma unroll
    for (int kt = 0; kt < H::KT; kt++)
      s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[cc & 1][kt], st.q[cc], cc == 0 ? st.negm : s[kt], 0, 0, 0);
  }
}

// Mask (tail: the block reaches past the sequence end), online-softmax statistics, P^T chunk by
// chunk and O^T += V^T P^T, for keys [k0, k0 + HK) of block kb.
//  * The running max moves only when the new max exceeds it by 2^8, so P <= 2^8 (exact).
//  * Accumulator elements 8*(j&1)..+7 of S^T group j/2 are keys 16j + 8h + 0..7: the B operand
//    of 16-key chunk j.
//  * V^T operand: within each 16-lane group, source lane 4r+c reads V[key0 + r][d0 + 4c .. +3];
//    the transpose read hands lane i the four keys key0..key0+3 at head-dim d0 + i.
//  * Masked keys: past the sequence end (one-dimensional blocks: only the last block), or, in
//    the PSABlock-centric layout (PAD), every position whose bit in the tile's validity words
//    (lo: positions 0..63, hi: 64..127) is clear -- 3D padding and the end of the sequence.
template <int D, int BLK, bool PAD>
__device__ __forceinline__ void softmax_pv_half(WaveState<D, BLK>& st,
                                                f32x16 (&s)[Half<D, BLK>::KT], const uint8_t* sv,
                                                int kb, int k0, int n, bool tail, uint64_t lo,
                                                uint64_t hi, int lane) {
  using T = Tile<D, BLK>;
  using H = Half<D, BLK>;
  const int h = lane >> 5, g = lane >> 4, j16 = lane & 15;
  if (tail) {
    asm volatile("" ::: "memory");        // keep the mask a branch taken only by partial tiles
    if constexpr (PAD) {
#pragma unroll
      for (int kt = 0; kt < H::KT; kt++) {
        // This lane's keys of group kt are positions r0 + {0..7, 16..23}: one 64-bit word.
        const int r0 = k0 + 32 * kt + 8 * h;
        const uint32_t win = (uint32_t)((r0 < 64 ? lo : hi) >> (r0 & 63));
#pragma unroll
        for (int i = 0; i < 16; i++)
          if (!((win >> (16 * (i >> 3) + (i & 7))) & 1u)) s[kt][i] = -__builtin_inff();
      }
    } else {
      const int kbase = kb * BLK + k0 + 8 * h;
#pragma unroll
      for (int kt = 0; kt < H::KT; kt++)
#pragma unroll
        for (int i = 0; i < 16; i++)
          if (kbase + kt * 32 + 16 * (i >> 3) + (i & 7) >= n) s[kt][i] = -__builtin_inff();
    }
  }

  // s holds S - base with base = -negm (the running max, or 0 before the first kept key).
  // The softmax and its P V form the longest dependent chain of a block; while a wave runs it,
  // it issues ahead of the other wave on its SIMD, whose Q K^T MFMAs fill the gaps (measured:
  // 3 % faster sparse, 2-4 % dense).
  __builtin_amdgcn_s_setprio(1);
  // Row max as four independent chains, then combined (a short dependent chain).
  float m4[4] = {-__builtin_inff(), -__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
#pragma unroll
  for (int kt = 0; kt < H::KT; kt++)
#pragma unroll
    for (int i = 0; i < 16; i++) m4[i & 3] = fmaxf(m4[i & 3], s[kt][i]);
  const float mx = fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3]));
  const float base = -st.negm[0];
  const float ms = pair_max(mx) + base;
  const bool need = ms - st.m > 8.0f;     // false for -inf - -inf (NaN)
  if (__builtin_amdgcn_ballot_w64(need)) {
    asm volatile("" ::: "memory");        // keep this rare path a branch
    const float alpha = need ? __builtin_amdgcn_exp2f(st.m - ms) : 1.0f;
    const float shift = need ? ms - base : 0.0f;
    st.m = need ? ms : st.m;
    st.l *= alpha;
#pragma unroll
    for (int dt = 0; dt < T::DT; dt++) st.o[dt] *= alpha;
#pragma unroll
    for (int kt = 0; kt < H::KT; kt++) s[kt] -= shift;
    const float nb = st.m == -__builtin_inff() ? 0.0f : -st.m;
#pragma unroll
    for (int i = 0; i < 16; i++) st.negm[i] = nb;
  }

  const int vkey = k0 + 8 * h + (j16 >> 2);
  const int vsw0 = swz<T::CPR>(vkey), vsw1 = swz<T::CPR>(vkey + 4);   // identical for vkey + 16 j
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int j = 0; j < H::KC; j++) {
    // The V^T operands of this chunk are read ahead of its exponentials, which hide the LDS
    // latency.
    bf16x8 va[T::DT];
#pragma unroll
    for (int dt = 0; dt < T::DT; dt++) {
      const int dd = dt * 32 + 16 * (g & 1) + 4 * (j16 & 3);
      const int lchunk = dd >> 3, inoff = (dd & 7) * 2;
      const uint8_t* a0 = sv + (vkey + 16 * j) * T::RB + ((lchunk ^ vsw0) << 4) + inoff;
      const uint8_t* a1 = sv + (vkey + 16 * j + 4) * T::RB + ((lchunk ^ vsw1) << 4) + inoff;
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((PSA_LDS s16x4*)a0);
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((PSA_LDS s16x4*)a1);
      va[dt] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
    __builtin_amdgcn_sched_barrier(0);      // keep the reads ahead of the exponentials
    f32x8 e;
#pragma unroll
    for (int x = 0; x < 8; x++) e[x] = __builtin_amdgcn_exp2f(s[j >> 1][8 * (j & 1) + x]);
    const bf16x8 p = __builtin_convertvector(e, bf16x8);
    // Row sum of the rounded weights, two per instruction: the normaliser matches the P that
    // multiplies V.
    st.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 0, 1), ones, st.l, false);
    st.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 2, 3), ones, st.l, false);
    st.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 4, 5), ones, st.l, false);
    st.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 6, 7), ones, st.l, false);
#pragma unroll
    for (int dt = 0; dt < T::DT; dt++)
      st.o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[dt], p, st.o[dt], 0, 0, 0);
  }
  __builtin_amdgcn_s_setprio(0);
}

// One key/value block with a single K and a single V buffer per workgroup, loaded by halves
// (BLK/2 keys) and three barriers per block:
//   QK(lo)          | wait V_lo(i), K_hi(i); barrier b1; load K_lo(i+1)
//   softmax+PV(lo), QK(hi) | wait V_hi(i);   barrier b2; load V_lo(i+1), K_hi(i+1)
//   softmax+PV(hi)  | wait K_lo(i+1);        barrier b3; load V_hi(i+1)
// A half is loaded at the first barrier after its last reader and awaited at the last barrier
// before its first reader, so every load is in flight for two or three phases.  Each wait leaves
// the loads issued after the awaited ones in flight (HW per half); the last block issues none.
template <int D, int BLK, bool PAD>
__device__ __forceinline__ void block_step(WaveState<D, BLK>& st, const DmaPlan<D, BLK>& plan,
                                           const __bf16* kh, const __bf16* vh, int kb, int kb_next,
                                           bool more, int n, const uint8_t* sk, const uint8_t* sv,
                                           const uint64_t* masks, int lane) {
  uint64_t lo = ~0ull, hi = ~0ull;
  bool tail;
  if constexpr (PAD) {
    const int kbu = __builtin_amdgcn_readfirstlane(kb);
    lo = masks[2 * kbu];
    hi = masks[2 * kbu + 1];
    tail = (lo & hi) != ~0ull;
  } else {
    tail = (kb + 1) * BLK > n;
  }
  using H = Half<D, BLK>;
  constexpr int HW = DmaPlan<D, BLK>::HW;
  f32x16 s[H::KT];
  qk_half<D, BLK>(st, s, sk, 0, lane);
  wait_dma<HW>();                                       // V_lo(i), K_hi(i); V_hi(i) may fly
  __syncthreads();
  if (more) issue_half<D, BLK>(plan, kh, plan.lds_k, 0, kb_next, n);
  softmax_pv_half<D, BLK, PAD>(st, s, sv, kb, 0, n, tail, lo, hi, lane);
  qk_half<D, BLK>(st, s, sk, H::HK, lane);
  if (more)                                             // V_hi(i); K_lo(i+1) may fly
    wait_dma<HW>();
  else
    wait_dma<0>();
  __syncthreads();
  if (more) {
    issue_half<D, BLK>(plan, vh, plan.lds_v, 0, kb_next, n);
    issue_half<D, BLK>(plan, kh, plan.lds_k, 1, kb_next, n);
  }
  softmax_pv_half<D, BLK, PAD>(st, s, sv, kb, H::HK, n, tail, lo, hi, lane);
  if (more) {
    wait_dma<2 * HW>();                                 // K_lo(i+1); V_lo, K_hi(i+1) may fly
    __syncthreads();
    issue_half<D, BLK>(plan, vh, plan.lds_v, 1, kb_next, n);
  }
}

// One work item: query block qb of one (batch, head).  `list` holds the kept key blocks in
// ascending order (SPARSE) or is ignored (dense: every block 0..nkv-1).  PAD: the sequence is
// the PSABlock-centric layout and `masks` holds the valid positions of every tile.
template <int D, int BLK, bool SPARSE, bool PAD = false>
__device__ __forceinline__ void process_item(const DmaPlan<D, BLK>& plan,
                                             const __bf16* __restrict__ qh,
                                             const __bf16* __restrict__ kh,
                                             const __bf16* __restrict__ vh,
                                             __bf16* __restrict__ oh, float* __restrict__ lseh,
                                             int n, int qb, int nkv, const uint16_t* list,
                                             float c, const uint8_t* sk, const uint8_t* sv,
                                             const uint64_t* masks = nullptr) {
  using T = Tile<D, BLK>;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, r32 = lane & 31;
  const int row = qb * BLK + wave * 32 + r32;

  WaveState<D, BLK> st;
  {
    const bf16x8* src = (const bf16x8*)(qh + (size_t)min(row, n - 1) * D) + h;
#pragma unroll
    for (int cc = 0; cc < T::DC; cc++) st.q[cc] = src[2 * cc];
    // Scaling consumes the Q registers here: the compiler then waits for these loads once,
    // before any K/V DMA is issued, instead of inside the block loop where the hardware counter
    // also counts the in-flight DMA.
#pragma unroll
    for (int cc = 0; cc < T::DC; cc++)
      st.q[cc] = __builtin_convertvector(__builtin_convertvector(st.q[cc], f32x8) * c, bf16x8);
#pragma unroll
    for (int cc = 0; cc < T::DC; cc++) asm volatile("" ::"v"(st.q[cc]));
  }
  st.m = -__builtin_inff();
  st.l = 0.0f;
  st.negm = (f32x16){};
#pragma unroll
  for (int dt = 0; dt < T::DT; dt++) st.o[dt] = (f32x16){};

  // Only the last block of a sequence can reach past its end, and it is always the last of an
  // ascending list.
  constexpr int HW = DmaPlan<D, BLK>::HW;
  if constexpr (SPARSE) {
    // Block indices are read from the list two steps ahead and kept in vector registers until
    // the step that issues their loads (issue_half takes the wave-uniform value), so no list
    // read waits on the path into the next Q K^T.
    int kb_v = 0, kb1_v = -1;
    if (nkv > 0) {
      kb_v = list[0];
      kb1_v = nkv > 1 ? (int)list[1] : -1;
      issue_half<D, BLK>(plan, kh, plan.lds_k, 0, kb_v, n);
      issue_half<D, BLK>(plan, vh, plan.lds_v, 0, kb_v, n);
      issue_half<D, BLK>(plan, kh, plan.lds_k, 1, kb_v, n);
      issue_half<D, BLK>(plan, vh, plan.lds_v, 1, kb_v, n);
      wait_dma<3 * HW>();                               // K_lo(0)
      __syncthreads();
    }
    for (int it = 0; it < nkv; it++) {
      const int kb2_v = it + 2 < nkv ? (int)list[it + 2] : -1;
      block_step<D, BLK, PAD>(st, plan, kh, vh, __builtin_amdgcn_readfirstlane(kb_v), kb1_v,
                              it + 1 < nkv, n, sk, sv, masks, lane);
      kb_v = kb1_v;
      kb1_v = kb2_v;
    }
  } else {
    if (nkv > 0) {
      issue_half<D, BLK>(plan, kh, plan.lds_k, 0, 0, n);
      issue_half<D, BLK>(plan, vh, plan.lds_v, 0, 0, n);
      issue_half<D, BLK>(plan, kh, plan.lds_k, 1, 0, n);
      issue_half<D, BLK>(plan, vh, plan.lds_v, 1, 0, n);
      wait_dma<3 * HW>();                               // K_lo(0)
      __syncthreads();
    }
    for (int it = 0; it < nkv; it++)
      block_step<D, BLK, PAD>(st, plan, kh, vh, it, it + 1 < nkv ? it + 1 : -1, it + 1 < nkv, n, sk,
                              sv, masks, lane);
  }

  // Epilogue: O = O^T / l, rows past the end are not stored.
  const float lsum = pair_sum(st.l);
  const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
  if (row < n) {
    __bf16* dst = oh + (size_t)row * D + 4 * h;
#pragma unroll
    for (int dt = 0; dt < T::DT; dt++)
#pragma unroll
      for (int a = 0; a < 4; a++) {
        const f32x4 v = {st.o[dt][4 * a] * inv, st.o[dt][4 * a + 1] * inv,
                         st.o[dt][4 * a + 2] * inv, st.o[dt][4 * a + 3] * inv};
        *(bf16x4*)(dst + dt * 32 + 8 * a) = __builtin_convertvector(v, bf16x4);
      }
    if (lseh && h == 0)
      lseh[row] = lsum > 0.0f ? (st.m + __builtin_log2f(lsum)) * 0.69314718055994530942f
                              : -__builtin_inff();
  }
}

// Whether a workspace holds a finished plan for exactly the sizes of this launch.
__device__ __forceinline__ bool plan_matches(const PlanHeader& h, const PlanHeader& e) {
  return h.magic == kPlanMagic && h.n_bh == e.n_bh && h.n_heads == e.n_heads && h.nb == e.nb &&
         h.block == e.block && h.n == e.n && h.frames == e.frames && h.height == e.height &&
         h.width == e.width && h.n_text == e.n_text && h.pbt == e.pbt && h.pbh == e.pbh &&
         h.pbw == e.pbw;
}

// Pops the next work item of the persistent schedule (one lane): from queue `queue` first, then
// from the others in turn; -1 once every queue is exhausted.  Queue x holds list positions
// queues[x] .. queues[x + 1] - 1 and the item at position i is order[i] (i itself without an
// order).  Counters only grow: a value at or past a queue's end is final, so an exhausted queue
// is recognised with a load and costs no atomic.
__device__ __forceinline__ int32_t pop_item(int32_t* __restrict__ queues,
                                            const int32_t* __restrict__ order, int& queue,
                                            int& exhausted) {
  while (exhausted < kNumQueues) {
    const int32_t start = queues[queue], len = queues[queue + 1] - start;
    int32_t* ctr = &queues[kQueueCounters + queue * kCounterStride];
    int32_t idx = len;
    if (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < len) idx = atomicAdd(ctr, 1);
    if (idx < len) return order ? order[start + idx] : start + idx;
    queue = (queue + 1) % kNumQueues;
    exhausted++;
  }
  return -1;
}

// Arms the queues of a dense call: n_items work items in their natural order, cut into
// kNumQueues contiguous ranges of (nearly) equal length, counters at zero.
__global__ __launch_bounds__(64) void psa_dense_arm_kernel(int32_t* __restrict__ queues,
                                                           int32_t n_items) {
  const int t = threadIdx.x;
  if (t <= kNumQueues) queues[t] = (int32_t)((int64_t)n_items * t / kNumQueues);
  if (t < kNumQueues) queues[kQueueCounters + t * kCounterStride] = 0;
}

// Re-arms the plan's queue counters before each run (a workspace without a matching plan is
// left alone).
__global__ __launch_bounds__(64) void psa_rearm_kernel(int32_t* __restrict__ queues,
                                                       const PlanHeader* __restrict__ header,
                                                       PlanHeader expect) {
  if (!plan_matches(*header, expect)) return;
  if (threadIdx.x < kNumQueues) queues[kQueueCounters + threadIdx.x * kCounterStride] = 0;
}

// Persistent sparse attention (two 4-wave workgroups per CU).  Workgroup w starts on queue w % kNumQueues (its XCD under
// round-robin dispatch) and moves on to the next queue when one runs dry, so every workgroup
// exits once all queues are exhausted.
template <int D, int BLK, bool PAD>
__global__ __launch_bounds__(BLK * 2) __attribute__((amdgpu_waves_per_eu(2, 2))) void psa_sparse_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    __bf16* __restrict__ o, float* __restrict__ lse, const psa_stripe_t* __restrict__ params,
    const int2* __restrict__ coords, const int32_t* __restrict__ order,
    int32_t* __restrict__ queues, const uint64_t* __restrict__ masks,
    const PlanHeader* __restrict__ header, PlanHeader expect, float c) {
  using T = Tile<D, BLK>;
  __shared__ __attribute__((aligned(1024))) uint8_t sk[T::BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sv[T::BYTES];
  __shared__ uint16_t list[PSA_MAX_BLOCKS];
  __shared__ int32_t misc[8];

  // A workspace without a finished plan for exactly these sizes is left alone: nothing is read
  // through its queues and no output is written.
  if (!plan_matches(*header, expect)) return;
  const int32_t n_heads = expect.n_heads, n = expect.n, nb = expect.nb;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  DmaPlan<D, BLK> plan;
  plan.init(lds_address(sk), lds_address(sv), __builtin_amdgcn_readfirstlane(wave), lane);
  int queue = blockIdx.x % kNumQueues, exhausted = 0;
  while (true) {
    if (tid == 0) misc[7] = pop_item(queues, order, queue, exhausted);
    __syncthreads();
    const int32_t item = misc[7];
    if (item < 0) break;
    const int32_t bh = item / nb, qb = item - bh * nb;
    const psa_stripe_t m = params[bh % n_heads];

    // In-kernel decode of the kept key blocks of this query block (ascending).
    const int2 cq = coords[qb];
    int32_t nkv = 0;
    for (int32_t base = 0; base < nb; base += T::kThreads) {
      const int32_t kb = base + tid;
      const bool keep = kb < nb && tile_keep(m, cq, coords[kb]);
      const uint64_t mask = __builtin_amdgcn_ballot_w64(keep);
      if (lane == 0) misc[wave] = __builtin_popcountll(mask);
      __syncthreads();
      int32_t pos = nkv, total = 0;
#pragma unroll
      for (int w = 0; w < T::kWaves; w++) {
        pos += w < wave ? misc[w] : 0;
        total += misc[w];
      }
      pos += __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                       __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
      if (keep) list[pos] = (uint16_t)kb;
      nkv += total;
      __syncthreads();
    }

    const size_t off = (size_t)bh * n * D;
    process_item<D, BLK, true, PAD>(plan, q + off, k + off, v + off, o + off,
                                    lse ? lse + (size_t)bh * n : nullptr, n, qb, nkv, list, c, sk,
                                    sv, masks);
  }
}

// Dense attention: one workgroup per (batch, head, query block); consecutive workgroups of one
// XCD (round-robin dispatch) take consecutive query blocks.
template <int D, int BLK>
__global__ __launch_bounds__(BLK * 2) __attribute__((amdgpu_waves_per_eu(2, 2))) void psa_dense_kernel(const __bf16* __restrict__ q,
                                                        const __bf16* __restrict__ k,
                                                        const __bf16* __restrict__ v,
                                                        __bf16* __restrict__ o,
                                                        float* __restrict__ lse, int32_t n,
                                                        int32_t nb, int32_t n_items,
                                                        int32_t* __restrict__ queues, float c) {
  using T = Tile<D, BLK>;
  __shared__ __attribute__((aligned(1024))) uint8_t sk[T::BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sv[T::BYTES];
  __shared__ int32_t next_item;
  DmaPlan<D, BLK> plan;
  plan.init(lds_address(sk), lds_address(sv), __builtin_amdgcn_readfirstlane(threadIdx.x >> 6),
            threadIdx.x & 63);
  int queue = blockIdx.x % kNumQueues, exhausted = 0;
  for (int round = 0;; round++) {
    int32_t item;
    if (queues) {
      // Persistent: items from the armed queues, this XCD's first, then the others'.
      if (threadIdx.x == 0) next_item = pop_item(queues, nullptr, queue, exhausted);
      __syncthreads();
      item = __builtin_amdgcn_readfirstlane(next_item);
      if (item < 0) break;
    } else {
      // One item per workgroup, consecutive workgroups of one XCD on consecutive items.
      if (round > 0) break;
      const int32_t per_xcd = gridDim.x / kNumQueues;
      item = (blockIdx.x % kNumQueues) * per_xcd + blockIdx.x / kNumQueues;
      if (item >= n_items) break;
    }
    const int32_t bh = item / nb, qb = item - bh * nb;
    const size_t off = (size_t)bh * n * D;
    process_item<D, BLK, false>(plan, q + off, k + off, v + off, o + off,
                                lse ? lse + (size_t)bh * n : nullptr, n, qb, nb, nullptr, c, sk, sv);
  }
}

// ---------------------------------------------------------------------------------------------
// Pair engine (BLK = 128): one workgroup of eight waves per CU.  Waves 0-3 take the first query
// block of a work item, waves 4-7 the second (each wave 32 rows, the per-wave tile engine
// above).  The two rows share one stream of K/V blocks -- the union of their kept sets, each
// entry marked with the rows that keep it -- double-buffered in LDS with one barrier per block
// and every block's loads issued during the block before (K after its barrier, V after its
// first Q K^T half); a row skips the blocks it does not keep.
// The plan pairs rows with equal kept sets, so a K/V block is loaded once for two query blocks
// and most entries are used by both rows.  Each row visits each of its own kept blocks once,
// with the one-row engine's arithmetic; the stream runs cyclically from a block the plan chooses
// (psa_starts_kernel), and from block 0 for pairs that keep every block.
// ---------------------------------------------------------------------------------------------

// Direct global->LDS loads of a whole K or V block by the eight waves of a workgroup: wave w
// loads the 1 KB slots w S .. w S + S - 1, with the row/chunk mapping and swizzle of DmaPlan.
template <int D, int BLK>
struct DmaPlan8 {
  using T = Tile<D, BLK>;
  static constexpr int S = T::BYTES / (1024 * 8);      // slots per wave per tensor
  static_assert(S >= 1 && T::BYTES % (1024 * 8) == 0, "tile shape");
  uint32_t off[S];
  int wave, lane;

  __device__ __forceinline__ void init(int wave_, int lane_) {
    wave = wave_;
    lane = lane_;
#pragma unroll
    for (int i = 0; i < S; i++) off[i] = offset(i, BLK);
  }

  // Byte offset in the block of the 16 bytes this lane loads for slot i; rows at or past `rows`
  // are clamped to row rows - 1 (their scores are masked).
  __device__ __forceinline__ uint32_t offset(int i, int rows) const {
    const int p = (wave * S + i) * 64 + lane;
    const int row = p / T::CPR;
    const int chunk = (p % T::CPR) ^ swz<T::CPR>(row);
    return (uint32_t)(min(row, rows - 1) * T::RB + chunk * 16);
  }
};

// Loads block kb of one tensor.  Waves 0-3 hold rows 0 .. BLK/2-1 and write them at lds_lo,
// waves 4-7 the upper rows at lds_hi (equal to lds_lo + BYTES/2 for a contiguous block, or a
// separate half-block buffer).
template <int D, int BLK>
__device__ __forceinline__ void issue_block8(const DmaPlan8<D, BLK>& plan, const __bf16* xh,
                                             uint32_t lds_lo, uint32_t lds_hi, int kb, int n) {
  using P = DmaPlan8<D, BLK>;
  using T = Tile<D, BLK>;
  kb = __builtin_amdgcn_readfirstlane(kb);
  const int rows = n - kb * BLK;
  const void* base = (const void*)(xh + (size_t)kb * BLK * D);
  const uint32_t dst = plan.wave < 4 ? lds_lo : lds_hi - (uint32_t)(T::BYTES / 2);
  const uint32_t l0 = __builtin_amdgcn_readfirstlane(dst + (uint32_t)(plan.wave * P::S) * 1024u);
  if (rows >= BLK) {
#pragma unroll
    for (int i = 0; i < P::S; i++) dma16(l0 + i * 1024u, plan.off[i], base);
  } else {
#pragma unroll
    for (int i = 0; i < P::S; i++) dma16(l0 + i * 1024u, plan.offset(i, rows), base);
  }
}

// O = O^T / l of a finished row block (rows past the end are not stored), LSE if asked.
template <int D, int BLK>
__device__ __forceinline__ void store_rows(const WaveState<D, BLK>& st, __bf16* __restrict__ oh,
                                           float* __restrict__ lseh, int row, int n, int lane) {
  using T = Tile<D, BLK>;
  const int h = lane >> 5;
  const float lsum = pair_sum(st.l);
  const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
  if (row < n) {
    __bf16* dst = oh + (size_t)row * D + 4 * h;
#pragma unroll
    for (int dt = 0; dt < T::DT; dt++)
#pragma unroll
      for (int a = 0; a < 4; a++) {
        const f32x4 v = {st.o[dt][4 * a] * inv, st.o[dt][4 * a + 1] * inv,
                         st.o[dt][4 * a + 2] * inv, st.o[dt][4 * a + 3] * inv};
        *(bf16x4*)(dst + dt * 32 + 8 * a) = __builtin_convertvector(v, bf16x4);
      }
    if (lseh && h == 0)
      lseh[row] = lsum > 0.0f ? (st.m + __builtin_log2f(lsum)) * 0.69314718055994530942f
                              : -__builtin_inff();
  }
}

// The same through LDS: the wave's 32 rows are staged row-major in `stage` (32 x 2D bytes of LDS
// no other wave touches; 16-byte chunks XOR-swizzled by the row), then stored as whole rows, 16
// bytes per lane, so that each store covers 64 x 16 contiguous bytes of O instead of 8 bytes in
// each of 32 rows.  row0 = the wave's first row; lane l holds row row0 + (l & 31).
template <int D, int BLK>
__device__ __forceinline__ void store_rows_staged(const WaveState<D, BLK>& st, __bf16* __restrict__ oh,
                                                  float* __restrict__ lseh, int row0, int n, int lane,
                                                  uint32_t stage) {
  using T = Tile<D, BLK>;
  constexpr int RB = 2 * D;                   // bytes per row
  constexpr int C16 = RB / 16;                // 16-byte chunks per row
  // The lane's addresses are formed here, not hoisted out of the item loop into registers that
  // would stay live across the block loop.
  asm volatile("" : "+v"(lane));
  const int h = lane >> 5, r = lane & 31;
  const float lsum = pair_sum(st.l);
  const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
#pragma unroll
  for (int dt = 0; dt < T::DT; dt++)
#pragma unroll
    for (int a = 0; a < 4; a++) {
      const f32x4 v = {st.o[dt][4 * a] * inv, st.o[dt][4 * a + 1] * inv,
                       st.o[dt][4 * a + 2] * inv, st.o[dt][4 * a + 3] * inv};
      const int chunk = (4 * dt + a) ^ (r & (C16 - 1));        // columns 8 (4 dt + a) + 4 h ...
      *(PSA_LDS bf16x4*)(uintptr_t)(stage + r * RB + chunk * 16 + 8 * h) = __builtin_convertvector(v, bf16x4);
    }
#pragma unroll 2
  for (int j = 0; j < 32 * C16 / 64; j++) {
    const int idx = 64 * j + lane, rr = idx / C16, c = idx % C16;
    const u32x4 val = *(PSA_LDS u32x4*)(uintptr_t)(stage + rr * RB + ((c ^ (rr & (C16 - 1))) * 16));
    if (row0 + rr < n) *(u32x4*)(oh + (size_t)(row0 + rr) * D + 8 * c) = val;
  }
  if (lseh && h == 0 && row0 + r < n)
    lseh[row0 + r] = lsum > 0.0f ? (st.m + __builtin_log2f(lsum)) * 0.69314718055994530942f
                                 : -__builtin_inff();
}

// Entry i of a pair's block stream: key block in bits 0-12, kept by the first row (bit 13) and
// by the second row (bit 14).
constexpr int kEntryRowShift = 13;
constexpr int kEntryBlockMask = (1 << kEntryRowShift) - 1;
static_assert(PSA_MAX_BLOCKS <= (1 << kEntryRowShift), "block index fits the entry");

// One work item of the pair engine: this wave's row (query block, -1: none) of one (batch, head)
// and nu stream entries (SPARSE: in `list`; dense: every block, kept by both rows).  Block i
// sits in buffer i & 1; after one barrier (its loads, issued a block earlier, have landed and
// block i - 1 is no longer read) the loads of block i + 1 go out and each row that keeps block
// i runs it: Q K^T, softmax and P V for each half.
template <int D, int BLK, bool SPARSE, bool PAD>
__device__ __forceinline__ void process_pair(const DmaPlan8<D, BLK>& plan, int grp,
                                             const __bf16* __restrict__ qh,
                                             const __bf16* __restrict__ kh,
                                             const __bf16* __restrict__ vh,
                                             __bf16* __restrict__ oh, float* __restrict__ lseh,
                                             int n, int my_row, int nu, int first,
                                             const uint16_t* list, float c,
                                             uint8_t (*sk)[Tile<D, BLK>::BYTES],
                                             uint8_t (*sv)[Tile<D, BLK>::BYTES],
                                             const uint64_t* masks) {
  using T = Tile<D, BLK>;
  using H = Half<D, BLK>;
  constexpr int HALF = T::BYTES / 2;
  const int tid = threadIdx.x, lane = tid & 63, gw = (tid >> 6) & 3;
  const int h = lane >> 5, r32 = lane & 31;
  const int row = my_row * BLK + gw * 32 + r32;

  // Entry i of the stream: list entry first + i, cyclically.
  auto entry = [&](int i) {
    if constexpr (SPARSE) {
      int j = i + first;
      j = j >= nu ? j - nu : j;
      return (int)__builtin_amdgcn_readfirstlane(list[j]);
    } else {
      return i | (3 << kEntryRowShift);
    }
  };
  auto issue_k = [&](int buf, int kb) {
    issue_block8<D, BLK>(plan, kh, lds_address(sk[buf]), lds_address(sk[buf]) + HALF, kb, n);
  };
  auto issue_v = [&](int buf, int kb) {
    issue_block8<D, BLK>(plan, vh, lds_address(sv[buf]), lds_address(sv[buf]) + HALF, kb, n);
  };
  int e = 0;
  // Sparse: the first block's loads go out before the Q loads, so that the two latencies overlap
  // at the start of the item (dense: after them; the other order measured slower there).
  if constexpr (SPARSE) {
    if (nu > 0) {
      e = entry(0);
      issue_k(0, e & kEntryBlockMask);
      issue_v(0, e & kEntryBlockMask);
    }
  }

  WaveState<D, BLK> st;
  if (my_row >= 0) {
    const bf16x8* src = (const bf16x8*)(qh + (size_t)min(row, n - 1) * D) + h;
#pragma unroll
    for (int cc = 0; cc < T::DC; cc++) st.q[cc] = src[2 * cc];
#pragma unroll
    for (int cc = 0; cc < T::DC; cc++)
      st.q[cc] = __builtin_convertvector(__builtin_convertvector(st.q[cc], f32x8) * c, bf16x8);
#pragma unroll
    for (int cc = 0; cc < T::DC; cc++) asm volatile("" ::"v"(st.q[cc]));
  }
  st.m = -__builtin_inff();
  st.l = 0.0f;
  st.negm = (f32x16){};
#pragma unroll
  for (int dt = 0; dt < T::DT; dt++) st.o[dt] = (f32x16){};

  if constexpr (!SPARSE) {
    if (nu > 0) {
      e = entry(0);
      issue_k(0, e & kEntryBlockMask);
      issue_v(0, e & kEntryBlockMask);
    }
  }
  for (int i = 0; i < nu; i++) {
    const int kb = e & kEntryBlockMask;
    const bool mine = my_row >= 0 && ((e >> (kEntryRowShift + grp)) & 1);
    uint64_t lo = ~0ull, hi = ~0ull;
    bool tail;
    if constexpr (PAD) {
      lo = masks[2 * kb];
      hi = masks[2 * kb + 1];
      tail = (lo & hi) != ~0ull;
    } else {
      tail = (kb + 1) * BLK > n;
    }
    wait_dma<0>();                                        // block i, issued a block ago
    __syncthreads();                                      // ... by every wave; block i-1 read
    // The next block's K goes out right after the barrier and its V after this block's first
    // Q K^T half: a wave stalls while it issues, and a single burst of all its loads after the
    // barrier, where every wave issues at once, keeps the MFMA pipes idle for longer (measured:
    // sparse 0.5-1.3 % and dense 0.4-3 % faster on two boxes, same bits).
    const bool more = i + 1 < nu;
    int kbn = 0;
    if (more) {
      e = entry(i + 1);
      kbn = e & kEntryBlockMask;
      issue_k((i + 1) & 1, kbn);
    }
    if (mine) {
      const uint8_t* skb = sk[i & 1];
      const uint8_t* svb = sv[i & 1];
      f32x16 s[H::KT];
      qk_half<D, BLK>(st, s, skb, 0, lane);
      if (more) issue_v((i + 1) & 1, kbn);
      softmax_pv_half<D, BLK, PAD>(st, s, svb, kb, 0, n, tail, lo, hi, lane);
      qk_half<D, BLK>(st, s, skb, H::HK, lane);
      softmax_pv_half<D, BLK, PAD>(st, s, svb, kb, H::HK, n, tail, lo, hi, lane);
    } else if (more) {
      issue_v((i + 1) & 1, kbn);
    }
  }
  if constexpr (SPARSE) {
    // The buffer of block nu - 2 (every wave passed the barrier of block nu - 1) stages the
    // output: 8 KB per wave, K half for group 0, V half for group 1.
    if (my_row >= 0) {
      static_assert(4 * 32 * 2 * D <= T::BYTES, "a wave's rows fit its share of a free buffer");
      const uint32_t stage = lds_address(grp == 0 ? sk[nu & 1] : sv[nu & 1]) + gw * (32 * 2 * D);
      store_rows_staged<D, BLK>(st, oh, lseh, my_row * BLK + gw * 32, n, lane, stage);
    }
  } else {
    if (my_row >= 0) store_rows<D, BLK>(st, oh, lseh, row, n, lane);
  }
}

// SPARSE: persistent, one workgroup per CU popping pair items from the plan's queues.  Dense: the
// pairs (2 p, 2 p + 1) of the flattened (batch*head, pair) list, either popped from armed queues
// by a persistent grid (queues given) or one pair per workgroup, consecutive workgroups of one
// XCD taking consecutive pairs.
// Byte offsets of the plan's sections in the workspace handed to the pair engine (a workspace of
// up to 4 GiB: one base pointer and 32-bit offsets keep fewer kernel arguments live in scalar
// registers than one pointer per section).
struct PlanView {
  uint32_t params, coords, order, queues, masks, pairs, starts;
};

template <int D, int BLK, bool SPARSE, bool PAD>
__global__ __launch_bounds__(BLK * 4) __attribute__((amdgpu_waves_per_eu(2, 2))) void psa_pair_kernel(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    __bf16* __restrict__ o, float* __restrict__ lse, const uint8_t* __restrict__ ws, PlanView pv,
    PlanHeader expect, float c) {
  using T = Tile<D, BLK>;
  const PlanHeader* header = (const PlanHeader*)ws;
  const psa_stripe_t* params = (const psa_stripe_t*)(ws + pv.params);
  const int2* coords = (const int2*)(ws + pv.coords);
  const int32_t* order = (const int32_t*)(ws + pv.order);
  int32_t* queues = ws ? (int32_t*)(ws + pv.queues) : nullptr;
  const uint64_t* masks = (const uint64_t*)(ws + pv.masks);
  const int2* pairs = (const int2*)(ws + pv.pairs);
  const int32_t* starts = (const int32_t*)(ws + pv.starts);
  static_assert(T::kWaves == 4, "a row is four waves");
  __shared__ __attribute__((aligned(1024))) uint8_t sk[2][T::BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sv[2][T::BYTES];
  __shared__ uint16_t list[SPARSE ? PSA_MAX_BLOCKS : 1];
  __shared__ int32_t misc[24];

  if constexpr (SPARSE) {
    // A workspace without a finished plan for exactly these sizes is left alone.
    if (!plan_matches(*header, expect)) return;
  }
  const int32_t n_heads = expect.n_heads, n = expect.n, nb = expect.nb;
  const int32_t np = pairs_per_head(nb), n_items = expect.n_bh * np;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int grp = __builtin_amdgcn_readfirstlane(wave >> 2);
  DmaPlan8<D, BLK> plan;
  plan.init(__builtin_amdgcn_readfirstlane(wave), lane);
  int queue = blockIdx.x % kNumQueues, exhausted = 0;
  for (int round = 0;; round++) {
    int32_t item;
    if constexpr (SPARSE) {
      if (tid == 0) misc[15] = pop_item(queues, order, queue, exhausted);
      __syncthreads();
      item = __builtin_amdgcn_readfirstlane(misc[15]);
      if (item < 0) break;
    } else if (queues) {
      // Dense, persistent: items from the armed queues in their natural order.
      if (tid == 0) misc[15] = pop_item(queues, nullptr, queue, exhausted);
      __syncthreads();
      item = __builtin_amdgcn_readfirstlane(misc[15]);
      if (item < 0) break;
    } else {
      // Dense, one item per workgroup, consecutive workgroups of one XCD on consecutive items.
      if (round > 0) break;
      const int32_t per_xcd = gridDim.x / kNumQueues;
      item = (blockIdx.x % kNumQueues) * per_xcd + blockIdx.x / kNumQueues;
      if (item >= n_items) break;
    }
    const int32_t bh = item / np, p = item - bh * np, h = bh % n_heads;
    int2 pr;
    if constexpr (SPARSE) {
      pr = pairs[(int64_t)h * np + p];
    } else {
      pr = make_int2(2 * p, 2 * p + 1 < nb ? 2 * p + 1 : -1);
    }
    const int my_row = __builtin_amdgcn_readfirstlane(grp == 0 ? pr.x : pr.y);

    int32_t nu = nb, first = 0;
    if constexpr (SPARSE) {
      // In-kernel decode of the union of the two rows' kept key blocks (ascending), and the
      // number of them below the block the plan starts this item's stream at (the stream then
      // runs cyclically from there).
      const psa_stripe_t m = params[h];
      const int2 ca = coords[pr.x];
      const int2 cb = pr.y >= 0 ? coords[pr.y] : make_int2(kDeadTile, 0);
      const int32_t start = starts[item];
      nu = 0;
      for (int32_t base = 0; base < nb; base += 8 * 64) {
        const int32_t kb = base + tid;
        const int2 ck = kb < nb ? coords[kb] : make_int2(kDeadTile, 0);
        const bool ka = tile_keep(m, ca, ck), kbk = tile_keep(m, cb, ck);
        const bool keep = ka || kbk;
        const uint64_t mask = __builtin_amdgcn_ballot_w64(keep);
        const uint64_t below = __builtin_amdgcn_ballot_w64(keep && kb < start);
        if (lane == 0) {
          misc[wave] = __builtin_popcountll(mask);
          misc[16 + wave] = __builtin_popcountll(below);
        }
        __syncthreads();
        int32_t pos = nu, total = 0;
#pragma unroll
        for (int w = 0; w < 8; w++) {
          pos += w < wave ? misc[w] : 0;
          total += misc[w];
          first += misc[16 + w];
        }
        pos += __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                         __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
        if (keep)
          list[pos] = (uint16_t)(kb | ((ka ? 1 : 0) << kEntryRowShift) | ((kbk ? 1 : 0) << (kEntryRowShift + 1)));
        nu += total;
        __syncthreads();
      }
      first = __builtin_amdgcn_readfirstlane(first < nu ? first : 0);
    }
    const size_t off = (size_t)bh * n * D;
    process_pair<D, BLK, SPARSE, PAD>(plan, grp, q + off, k + off, v + off, o + off,
                                      lse ? lse + (size_t)bh * n : nullptr, n, my_row, nu, first, list,
                                      c, sk, sv, masks);
  }
}

template <int D, int BLK, bool PAD>
static hipError_t launch_sparse_t(const void* q, const void* k, const void* v, void* o,
                                  float* lse, const PlanHeader& expect, float c,
                                  void* workspace, const WorkspaceLayout& wl, int32_t n_wg,
                                  hipStream_t stream, bool rearm) {
  char* ws = (char*)workspace;
  if (rearm) {
    hipLaunchKernelGGL(psa_rearm_kernel, dim3(1), dim3(64), 0, stream, (int32_t*)(ws + wl.queues),
                       (const PlanHeader*)(ws + wl.header), expect);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if constexpr (BLK == 128) {
    // one eight-wave pair workgroup per CU
    static_assert(sizeof(PlanHeader) <= 256, "the plan header is the workspace's first section");
    const PlanView pv = {(uint32_t)wl.params, (uint32_t)wl.coords, (uint32_t)wl.order, (uint32_t)wl.queues,
                         (uint32_t)(PAD ? wl.masks : 0), (uint32_t)wl.pairs, (uint32_t)wl.starts};
    hipLaunchKernelGGL((psa_pair_kernel<D, BLK, true, PAD>), dim3(n_wg / 2), dim3(4 * BLK), 0, stream,
                       (const __bf16*)q, (const __bf16*)k, (const __bf16*)v, (__bf16*)o, lse,
                       (const uint8_t*)ws, pv, expect, c);
  } else {
    hipLaunchKernelGGL((psa_sparse_kernel<D, BLK, PAD>), dim3(n_wg), dim3(Tile<D, BLK>::kThreads), 0, stream,
                       (const __bf16*)q, (const __bf16*)k, (const __bf16*)v, (__bf16*)o, lse,
                       (const psa_stripe_t*)(ws + wl.params), (const int2*)(ws + wl.coords),
                       (const int32_t*)(ws + wl.order), (int32_t*)(ws + wl.queues),
                       PAD ? (const uint64_t*)(ws + wl.masks) : nullptr,
                       (const PlanHeader*)(ws + wl.header), expect, c);
  }
  return hipGetLastError();
}

hipError_t launch_sparse(const void* q, const void* k, const void* v, void* o, float* lse,
                         int32_t batch, int32_t n_heads, int32_t head_dim, const Geometry& g,
                         float c, void* workspace, const WorkspaceLayout& wl, int32_t n_wg,
                         hipStream_t stream, bool rearm) {
  const PlanHeader e = plan_header(g, batch, n_heads);
  if (g.pbt > 0) {
    if (head_dim == 128 && g.block == 128)
      return launch_sparse_t<128, 128, true>(q, k, v, o, lse, e, c, workspace, wl, n_wg, stream, rearm);
    if (head_dim == 64 && g.block == 64)
      return launch_sparse_t<64, 64, true>(q, k, v, o, lse, e, c, workspace, wl, n_wg, stream, rearm);
    if (head_dim == 128 && g.block == 64)
      return launch_sparse_t<128, 64, true>(q, k, v, o, lse, e, c, workspace, wl, n_wg, stream, rearm);
    if (head_dim == 64 && g.block == 128)
      return launch_sparse_t<64, 128, true>(q, k, v, o, lse, e, c, workspace, wl, n_wg, stream, rearm);
    return hipErrorInvalidValue;
  }
  if (head_dim == 128 && g.block == 128)
    return launch_sparse_t<128, 128, false>(q, k, v, o, lse, e, c, workspace, wl, n_wg, stream, rearm);
  if (head_dim == 64 && g.block == 64)
    return launch_sparse_t<64, 64, false>(q, k, v, o, lse, e, c, workspace, wl, n_wg, stream, rearm);
  if (head_dim == 128 && g.block == 64)
    return launch_sparse_t<128, 64, false>(q, k, v, o, lse, e, c, workspace, wl, n_wg, stream, rearm);
  if (head_dim == 64 && g.block == 128)
    return launch_sparse_t<64, 128, false>(q, k, v, o, lse, e, c, workspace, wl, n_wg, stream, rearm);
  return hipErrorInvalidValue;
}

// Dense attention.  With queues (a dense workspace) a one-thread-group kernel arms them and a
// persistent grid of n_wg one-row workgroups (n_wg / 2 pair workgroups) takes the items;
// without, one workgroup per item.
template <int D, int BLK>
static hipError_t launch_dense_t(const void* q, const void* k, const void* v, void* o, float* lse,
                                 int32_t n_bh, int32_t n, float c, int32_t* queues, int32_t n_wg,
                                 hipStream_t stream) {
  const int32_t nb = (n + BLK - 1) / BLK;
  const int32_t n_items = BLK == 128 ? n_bh * pairs_per_head(nb) : n_bh * nb;
  const int32_t per_xcd = (n_items + kNumQueues - 1) / kNumQueues;
  if (queues) {
    hipLaunchKernelGGL(psa_dense_arm_kernel, dim3(1), dim3(64), 0, stream, queues, n_items);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if constexpr (BLK == 128) {
    PlanHeader e = {};
    e.n_bh = n_bh;
    e.n_heads = n_bh;
    e.nb = nb;
    e.n = n;
    const int32_t grid = queues ? n_wg / 2 : per_xcd * kNumQueues;
    const PlanView pv = {0, 0, 0, 0, 0, 0, 0};      // the dense workspace is the queue area
    hipLaunchKernelGGL((psa_pair_kernel<D, BLK, false, false>), dim3(grid), dim3(4 * BLK), 0, stream,
                       (const __bf16*)q, (const __bf16*)k, (const __bf16*)v, (__bf16*)o, lse,
                       (const uint8_t*)queues, pv, e, c);
  } else {
    const int32_t grid = queues ? n_wg : per_xcd * kNumQueues;
    hipLaunchKernelGGL((psa_dense_kernel<D, BLK>), dim3(grid), dim3(Tile<D, BLK>::kThreads), 0, stream,
                       (const __bf16*)q, (const __bf16*)k, (const __bf16*)v, (__bf16*)o, lse, n, nb,
                       n_items, queues, c);
  }
  return hipGetLastError();
}

hipError_t launch_dense(const void* q, const void* k, const void* v, void* o, float* lse,
                        int32_t batch, int32_t n_heads, int32_t head_dim, int32_t n_tokens,
                        int32_t block, float c, int32_t* queues, int32_t n_workgroups,
                        hipStream_t stream) {
  const int32_t n_bh = batch * n_heads;
  const int32_t w = n_workgroups;
  if (head_dim == 128 && block == 128)
    return launch_dense_t<128, 128>(q, k, v, o, lse, n_bh, n_tokens, c, queues, w, stream);
  if (head_dim == 64 && block == 64)
    return launch_dense_t<64, 64>(q, k, v, o, lse, n_bh, n_tokens, c, queues, w, stream);
  if (head_dim == 128 && block == 64)
    return launch_dense_t<128, 64>(q, k, v, o, lse, n_bh, n_tokens, c, queues, w, stream);
  if (head_dim == 64 && block == 128)
    return launch_dense_t<64, 128>(q, k, v, o, lse, n_bh, n_tokens, c, queues, w, stream);
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------------------------
// Static scratch of psa_attention_fwd_noalloc: the plan of a call lives in this array instead of
// a caller's workspace.  Every GPU the library runs on holds its own copy, from the time the
// library's code is loaded on it until the process ends.  In host code `scratch` names a host-side
// stand-in, not a device address: the kernels only ever get the address scratch_pointer() looked
// up for the current device.
// ---------------------------------------------------------------------------------------------

static __device__ __align__(256) uint8_t scratch[PSA_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 256;
std::mutex g_scratch_lock;
void* g_scratch_address[kMaxDevices];      // per device, once looked up
}  // namespace

hipError_t scratch_pointer(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_lock);
  if (!g_scratch_address[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));       // device `dev` is current
    if (e != hipSuccess) return e;
    if (!p || ((uintptr_t)p & 255) != 0) return hipErrorInvalidSymbol;
    g_scratch_address[dev] = p;
  }
  *out = g_scratch_address[dev];
  return hipSuccess;
}

}  // namespace psa
