// Internal declarations shared by the host runtime and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace bsa {

constexpr int kHeadDim = 128;

// One workgroup task (Section 4.3): a contiguous slice [tile_begin, tile_end)
// of the active KV tiles of physical query tile `pq` of head `bh`
// (= b * heads + h).  `split` is the slice's ordinal among the row's `nsplit`
// slices; nsplit > 1 means the row is reduced by Split-K.
struct Task {
  int32_t bh, pq, tile_begin, tile_end, split, nsplit, pad0, pad1;
};
static_assert(sizeof(Task) == 32, "Task is 32 bytes");

// Per-head facts for the mask kernels.
struct HeadDesc {
  int64_t mask_off;  // offset of the head's mask inside one batch
  int32_t nqb, nkb;  // logical block grid
  int32_t seg;       // geometry segment
  int32_t pad;
};

// Device-side statistics of one segment (integer atomics only).
struct SegStats {
  unsigned long long nnz, run_blocks, max_row_nnz, pad;
};

// A range of logical rows inside one (b, h), reduced by one workgroup.
struct RowChunk {
  int64_t begin, end;
  int32_t bh, seg;
};

struct MaskStateArgs {
  const uint8_t* mask;
  int64_t stride_b;
  const HeadDesc* heads;
  const int64_t* row_base;  // [B*H + 1], logical rows of (b, h) start here
  int32_t H, nbh;
  int64_t R;
  int32_t* counts;          // [R]   (count pass)
  int32_t* runs;            // [R]   (count pass) active blocks of the row in runs of length >= 2
  const RowChunk* chunks;   // [nchunks] (count pass) reduction ranges
  int32_t nchunks;
  const int64_t* row_ptr;   // [R+1] (fill pass)
  int32_t* col_idx;         // [nnz] (fill pass)
  SegStats* seg_stats;      // [nseg]
  unsigned long long* bh_nnz;  // [B*H]
  int32_t wide;             // every mask row starts 4-byte aligned and nkb % 4 == 0
};

struct MapArgs {
  const uint8_t* mask;
  int64_t stride_b;
  const HeadDesc* heads;
  const int32_t* seg_heads;  // heads of the segment, ascending
  int32_t nsh, H;
  int32_t npq, npk;          // physical grid of one head
  int32_t nqb, nkb;          // logical grid of one head
  int32_t gq, gkv, rq, rkv;  // members per tile / tiles per block along Q and KV
  int64_t Rp;                // physical rows of the segment = B * nsh * npq
  int32_t* counts;           // count pass
  const int64_t* tile_ptr;   // fill pass
  int32_t* tile_kv;
  uint64_t* member;          // may be null (no membership metadata)
  int32_t wide;              // mask rows 4-byte aligned and nkb % 4 == 0 (see MaskStateArgs)
};

struct TaskArgs {
  const int64_t* tile_ptr;   // physical (or, for Direct, logical) row offsets
  const int64_t* row_base;   // logical row base per (b, h); used when direct
  const int32_t* seg_heads;
  int32_t nsh, H, npq, split;
  int32_t direct;
  int64_t Rp;
  int32_t* counts;           // count pass (split > 1)
  const int64_t* task_ptr;   // fill pass (split > 1), null when split == 1
  Task* tasks;
};

// Dispatch order of a segment's tasks (task_order.hip): a permutation of the
// task indices, row order with every task moved up to the first task that
// has the same KV tile list (and member bits).  Work arrays are [ntasks].
struct OrderArgs {
  const Task* tasks;
  const int64_t* ntasks_dev;  // device task count (may be null)
  int64_t ntasks;             // exact count, or the bound when ntasks_dev is set
  const int32_t* tile_kv;
  const uint64_t* member;     // may be null
  uint64_t* table_key;        // [table_size] list hashes (0: free slot)
  int32_t* table_min;         // [table_size] lowest task index per hash
  int64_t table_size;         // a power of two >= 2 * ntasks
  int32_t* task_slot;         // table slot of each task
  int32_t* idx_in;
  uint32_t* rep;              // representative task of each task
  uint32_t* rep_sorted;
  int32_t* order;             // out; the first (device count) entries are the real tasks
  Task* tasks_out;            // out (may be null): tasks[order[i]] at i; only without a device count
  void* temp;
  size_t temp_bytes;
};

struct AttnArgs {
  const Task* tasks;
  int32_t ntasks;              // exact count, or an upper bound when ntasks_dev is set
  const int64_t* ntasks_dev;   // device count (may be null)
  const int32_t* order;        // dispatch order of the tasks (may be null: as built)
  const int32_t* kv_tile;
  const uint64_t* member;      // null: every tile is fully active
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;                  // may be null
  float* ws;                   // Split-K partial states (may be null when no row splits)
  const uint16_t* zero_page;   // 256 zero bytes, read for K/V rows past the sequence end
  int64_t qs0, qs1, qs2, ks0, ks1, ks2, vs0, vs1, vs2, os0, os1, os2;
  int32_t H, Nq, Nkv;
  int32_t bq_shift, bkv_shift;  // log2 of the logical block sizes
  int32_t gq, gkv;              // membership grid of a tile
  float scale_log2;             // log2(e) / sqrt(d)
  int32_t slot_group, slot_run; // launch-slot to task map: XCDs per group (1, 2, 4 or 8) and run length
  int32_t balanced;             // nonzero: group g's share of the task list is [share_lo[g], share_lo[g + 1])
  int32_t share_lo[5];
  int64_t nslots;               // launch slots (0: the task count rounded up to 8)
};

// Kernel launchers (defined in the .hip files).
hipError_t launch_mask_count(const MaskStateArgs& a, hipStream_t s);
hipError_t launch_mask_fill(const MaskStateArgs& a, hipStream_t s);
hipError_t launch_scan_i32(const int32_t* in, int64_t* out, int64_t n, int64_t* block_tmp, hipStream_t s);
int64_t scan_tmp_elems(int64_t n);
hipError_t launch_map_count(const MapArgs& a, hipStream_t s);
hipError_t launch_map_fill(const MapArgs& a, hipStream_t s);
hipError_t launch_task_count(const TaskArgs& a, hipStream_t s);
hipError_t launch_task_fill(const TaskArgs& a, hipStream_t s);
hipError_t launch_attention(int tq, int tkv, int waves, int stages, const AttnArgs& a, hipStream_t s);
int64_t task_order_table_size(int64_t n);
hipError_t task_order_temp_bytes(int64_t n, size_t* bytes);
hipError_t launch_task_order(const OrderArgs& a, hipStream_t s);
hipError_t launch_splitk_merge(int tq, const AttnArgs& a, hipStream_t s);

// Top-k sparsifier (sparsify.hip): block means of a [B, N, H, 128] bf16
// tensor for heads [bh0, bh0 + nbh) into out[nbh][ceil(N / blk)][128] (fp64),
// the score rows of those heads, and the uint8 mask rows they select.
int32_t sparsify_max_kv_blocks();
hipError_t launch_block_mean(const uint16_t* x, int64_t s0, int64_t s1, int64_t s2, int32_t H, int32_t n,
                             int32_t blk, int32_t bh0, int32_t nbh, double* out, hipStream_t s);
hipError_t launch_block_scores(const double* pq, const double* pk, int32_t nqb, int32_t nkb, int32_t nbh,
                               double* scores, hipStream_t s);
hipError_t launch_topk_select(const double* scores, int32_t nqb, int32_t nkb, int32_t k, int32_t diagonal,
                              int32_t nq, int32_t nkv, int32_t bq, int32_t bkv, int32_t bh0, int32_t nbh,
                              uint8_t* mask, hipStream_t s);


}  // namespace bsa
