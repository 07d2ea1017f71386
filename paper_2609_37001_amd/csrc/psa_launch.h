// Internal interface between the C ABI (psa_api.hip) and the kernels (psa_kernels.hip).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

#include "psa.h"

namespace psa {

// Number of work queues of the sparse scheduler: one per XCD of an MI355X (8 XCDs of 32 CUs).
constexpr int kNumQueues = 8;

// Heads whose stripe parameters travel in one kernel-argument block.
constexpr int kHeadsPerChunk = 64;

struct ParamChunk {
  int32_t n;                        // heads in this chunk
  psa_stripe_t m[kHeadsPerChunk];
};

// Sequence geometry in blocks.  With one-dimensional blocks (pbt = 0) a block is `block`
// consecutive tokens of the frame-major sequence.  With 3D PSABlocks (pbt > 0) the sequence is
// the PSABlock-centric layout: the padded grid ordered (T', H', W', bt, bh, bw), then the text
// tokens; a block (tile) is `block` consecutive positions of it, and a PSABlock is a whole
// number of tiles.
struct Geometry {
  int32_t hw;       // tokens per frame of the video grid, H*W
  int32_t n_video;  // F*H*W
  int32_t n;        // tokens of the sequence: n_video + n_text, or n_blk + n_text (3D)
  int32_t n_text;
  int32_t block;
  int32_t nb;       // ceil(n / block)
  int32_t frames, height, width;
  int32_t pbt, pbh, pbw;   // PSABlock shape; pbt = 0 for one-dimensional blocks
  int32_t tp, hp, wp;      // PSABlock grid T', H', W' (3D)
  int32_t n_blk;           // positions of the padded video grid, T'H'W' * pbt*pbh*pbw (3D)
};

// Coordinate of a tile that holds only padding: never kept as a key, no work as a query.
constexpr int32_t kDeadTile = -2;

// Identifies a finished plan in the workspace header; the sizes it was made for follow it.
constexpr uint32_t kPlanMagic = 0x50534131u;  // "PSA1"

struct PlanHeader {
  uint32_t magic;   // kPlanMagic once the plan's kernels have run, 0 while they run
  int32_t n_bh;     // batch * n_heads
  int32_t n_heads;
  int32_t nb;
  int32_t block;
  int32_t n;
  int32_t frames, height, width, n_text;
  int32_t pbt, pbh, pbw;
};

// Layout of the queue area (int32 words): kNumQueues + 1 boundaries in the first 128-byte line,
// then one pop counter per queue, each in a line of its own (device-scope atomics on one line
// are serialised).
constexpr int kCounterStride = 32;
constexpr int kQueueCounters = 32;
constexpr int kQueueWords = kQueueCounters + kNumQueues * kCounterStride;
// Word of the first line (after the boundaries) counting the finished workgroups of the plan's
// last kernel at block 128.
constexpr int kStartsDone = 16;
static_assert(kStartsDone > kNumQueues && kStartsDone < kQueueCounters, "free word of the first line");

// Workspace of psa_dense_fwd: the queue area alone, rounded up to 256 bytes.
constexpr size_t kDenseWorkspaceBytes = (sizeof(int32_t) * kQueueWords + 255) / 256 * 256;

// Workspace of psa_attention_plan / psa_attention_run (byte offsets, each 256-aligned).
struct WorkspaceLayout {
  size_t header;    // PlanHeader
  size_t params;    // psa_stripe_t [n_heads]
  size_t coords;    // int2 [nb]: (frame, slot) of each block, frame = -1 for a global block
  size_t counts;    // int32 [batch*n_heads*nb]: kept key blocks per work item
  size_t order;     // int32 [batch*n_heads*nb]: work items in schedule order
  size_t queues;    // int32 [kQueueWords]: queue boundaries and pop counters
  size_t sigs;      // uint64 [n_heads][nb]: signature of each query block's kept set
  size_t pairs;     // int2 [n_heads][ceil(nb/2)]: query blocks paired into one work item
  size_t spans;     // uint32 [batch*n_heads*ceil(nb/2)]: first and last kept non-global key block
                    // of each pair item (bits 0-15, 16-31; 0xffffffff: none)
  size_t runspans;  // uint32 [batch*n_heads*ceil(nb/2)]: union of the spans of the items of the
                    // item's run (its head's range in its queue; a long item alone)
  size_t starts;    // int32 [batch*n_heads*ceil(nb/2)]: key block each pair item's stream starts at
  size_t masks;     // uint64 [nb][2]: valid positions of each tile (3D only)
  size_t total;
};

// Query blocks of one head processed together by the pair engine (BLK = 128): ceil(nb / 2)
// pairs per head, the second member -1 for a single.
__host__ __device__ inline int32_t pairs_per_head(int32_t nb) { return (nb + 1) / 2; }

WorkspaceLayout workspace_layout(int32_t batch, int32_t n_heads, int32_t nb, bool masks);

// Launchers; each returns the hipError_t of its launch(es).
hipError_t launch_blockmap(const ParamChunk& pc, int32_t head0, const Geometry& g,
                           uint8_t* blockmap, int32_t* kept_per_row, int64_t* kept_per_head,
                           hipStream_t stream);

hipError_t launch_setup(const ParamChunk& pc, int32_t head0, const Geometry& g, void* workspace,
                        const WorkspaceLayout& wl, bool write_coords, hipStream_t stream);

// PSABlock-level block map: groups 0 .. T'H'W'-1 are the PSABlocks, group T'H'W' (with text)
// the text; g.nb must be the group count.
hipError_t launch_group_blockmap(const ParamChunk& pc, int32_t head0, const Geometry& g,
                                 uint8_t* blockmap, int32_t* kept_per_row, int64_t* kept_per_head,
                                 hipStream_t stream);

// Chunks per (batch, head) of the L2 distance's first pass.
constexpr int kL2Chunks = 64;

// Per (batch, head) sums of (o - ref)^2 and ref^2 over [tokens][d] bf16 rows: fp32 partial sums
// per chunk, combined in fp64 in a fixed order (partial: kL2Chunks * 2 doubles per row).
hipError_t launch_l2(const void* o, const void* ref, int32_t n_bh, int64_t elems_per_bh,
                     double* partial, double* sq_err, double* sq_ref, hipStream_t stream);

// PSABlock-centric layout of [bh][tokens][d] tensors (to: original -> blocked, else back).
hipError_t launch_layout(const void* src, void* dst, int32_t n_bh, int32_t head_dim,
                         const Geometry& g, bool to_blocks, hipStream_t stream);

// Counts the kept blocks of every work item, orders them, and writes the header last.
hipError_t launch_schedule(const Geometry& g, int32_t batch, int32_t n_heads, void* workspace,
                           const WorkspaceLayout& wl, int32_t* kept_per_row, hipStream_t stream);

hipError_t launch_sparse(const void* q, const void* k, const void* v, void* o, float* lse,
                         int32_t batch, int32_t n_heads, int32_t head_dim, const Geometry& g,
                         float scale_log2, void* workspace, const WorkspaceLayout& wl,
                         int32_t n_workgroups, hipStream_t stream, bool rearm = true);

// queues: the int32 [kQueueWords] queue area of a dense workspace (persistent grid of
// n_workgroups one-row workgroups), or nullptr (one workgroup per work item).
hipError_t launch_dense(const void* q, const void* k, const void* v, void* o, float* lse,
                        int32_t batch, int32_t n_heads, int32_t head_dim, int32_t n_tokens,
                        int32_t block, float scale_log2, int32_t* queues, int32_t n_workgroups,
                        hipStream_t stream);

// Device address of the static scratch of psa_attention_fwd_noalloc on the current device
// (PSA_NOALLOC_SCRATCH_BYTES, 256-byte aligned), looked up once per device.
hipError_t scratch_pointer(void** out);

}  // namespace psa
