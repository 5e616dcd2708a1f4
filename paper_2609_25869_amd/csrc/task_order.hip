// Dispatch order of a segment's tasks.
//
// The attention kernel hands the dispatch order to the XCDs in runs of
// consecutive tasks (each XCD group takes a contiguous share, its XCDs
// alternate runs of 8), and an XCD holds a few dozen tasks at once that all
// stream K/V tiles through its own L2.  Two tasks share L2 lines only if they read the
// same tile at nearly the same time, which in practice means their tile lists
// are equal and they start together.  In row order that happens only by
// chance: under a multi-dimensional window, query blocks with equal KV lists
// sit a grid stride apart, and tasks with shorter lists drift ahead of the
// others.  The order used here is row order, except that every task moves up
// to the first task (in row order) with the same KV tile list: equal lists
// are dispatched together, finish together, and hand their slots to the next
// group together, while rows whose lists are unique keep the row order, in
// which neighbouring rows usually read overlapping lists.  Every task still
// computes exactly what it computed before, so results do not change; a hash
// collision can only cost locality.
#include <utility>

#include "bsa_internal.h"

namespace bsa {

namespace {

// SplitMix64 finaliser (Steele, Lea and Flood, "Fast splittable
// pseudorandom number generators", OOPSLA 2014).
__device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

constexpr int kWavesPerBlock = 4;

// Hash of task t's (bh, tile count, tile list, member bits), one wave per
// task, entered into an open-addressing table that keeps, per distinct hash,
// the lowest task index (the representative).  The probe loop is bounded by
// the table size, which is at least twice the task count, so it always finds
// a free or matching slot.
__global__ __launch_bounds__(64 * kWavesPerBlock) void task_hash_kernel(OrderArgs a) {
  const int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= a.ntasks) return;
  const int64_t nt = a.ntasks_dev ? *a.ntasks_dev : a.ntasks;
  if (t >= nt) return;
  const Task tk = a.tasks[t];
  const int64_t n = (int64_t)tk.tile_end - tk.tile_begin;
  uint64_t h = 0;
  for (int64_t i = lane; i < n; i += 64) {
    const uint64_t kv = (uint32_t)a.tile_kv[tk.tile_begin + i];
    const uint64_t mem = a.member ? a.member[tk.tile_begin + i] : 0ull;
    h += mix64(kv | ((uint64_t)i << 32)) ^ mix64(mem + 0x9e3779b97f4a7c15ull * (uint64_t)(i + 1));
  }
  for (int off = 32; off > 0; off >>= 1) h += __shfl_xor(h, off);
  h = mix64(h ^ mix64(((uint64_t)(uint32_t)tk.bh << 32) | (uint64_t)(uint32_t)n));
  if (h == 0) h = 1;  // 0 marks a free slot
  if (lane == 0) {
    const uint64_t mask = (uint64_t)a.table_size - 1;
    uint64_t slot = h & mask;
    int32_t found = -1;  // stays -1 only if the table were full, which its size rules out
    for (int64_t probe = 0; probe < a.table_size; ++probe) {
      const unsigned long long prev = atomicCAS(reinterpret_cast<unsigned long long*>(a.table_key + slot), 0ull,
                                                (unsigned long long)h);
      if (prev == 0ull || prev == h) {
        atomicMin(a.table_min + slot, (int32_t)t);
        found = (int32_t)slot;
        break;
      }
      slot = (slot + 1) & mask;
    }
    a.task_slot[t] = found;
  }
}

__global__ __launch_bounds__(256) void table_clear_kernel(OrderArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.table_size) return;
  a.table_key[i] = 0ull;
  a.table_min[i] = INT32_MAX;
}

// Representative of each task (tasks past the device count represent
// themselves, so they sort behind every real task), and the identity as the
// values of the sort.
__global__ __launch_bounds__(256) void representative_kernel(OrderArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= a.ntasks) return;
  const int64_t nt = a.ntasks_dev ? *a.ntasks_dev : a.ntasks;
  const int32_t slot = t < nt ? a.task_slot[t] : -1;
  a.rep[t] = slot < 0 ? (uint32_t)t : (uint32_t)a.table_min[slot];
  a.idx_in[t] = (int32_t)t;
}

// The tasks themselves in dispatch order, so the kernel reads its task with
// no indirection (tasks without Split-K partners only: the merge finds the
// partial states of a row's pieces next to each other in row order).
__global__ __launch_bounds__(256) void task_gather_kernel(OrderArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= a.ntasks) return;
  a.tasks_out[t] = a.tasks[a.order[t]];
}

int rep_bits(int64_t n) {  // bits of the largest task index n - 1, at least 1
  int b = 1;
  while (b < 31 && (int64_t(1) << b) < n) ++b;
  return b;
}

unsigned grid(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

// ---- stable sort of (representative, task index) pairs by representative:
// least-significant-digit passes over 8-bit digits, each a stable counting
// sort.  A pass cuts the list into tiles of 256 pairs (one workgroup each):
// digit histograms per tile, an exclusive scan over (digit, tile) in
// digit-major order, and a scatter in which a pair's place is its digit's
// offset for its tile plus the number of pairs before it in the tile with
// the same digit.

constexpr int kSortTile = 256;
constexpr int kSortWaves = kSortTile / 64;

int sort_passes(int64_t n) { return (rep_bits(n) + 7) / 8; }

// digit histogram of every tile, written as hist[digit * ntiles + tile]
__global__ __launch_bounds__(kSortTile) void digit_hist_kernel(const uint32_t* keys, int64_t n, int shift,
                                                               int32_t* hist, int64_t ntiles) {
  __shared__ int32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * kSortTile + threadIdx.x;
  if (i < n) atomicAdd(&h[(keys[i] >> shift) & 255], 1);
  __syncthreads();
  hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[threadIdx.x];
}

// Stable scatter of one tile: the rank of a pair among the tile's pairs with
// the same digit comes from eight ballots per wave (the lanes whose digit
// agrees on every bit) and the counts of the waves before it.
__global__ __launch_bounds__(kSortTile) void digit_scatter_kernel(const uint32_t* keys_in, const int32_t* vals_in,
                                                                  int64_t n, int shift, const int64_t* offsets,
                                                                  int64_t ntiles, uint32_t* keys_out,
                                                                  int32_t* vals_out) {
  __shared__ int32_t wave_count[kSortWaves][256];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  for (int j = threadIdx.x; j < kSortWaves * 256; j += kSortTile) (&wave_count[0][0])[j] = 0;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * kSortTile + threadIdx.x;
  const bool valid = i < n;
  const uint32_t key = valid ? keys_in[i] : 0u;
  const int d = (int)((key >> shift) & 255);
  uint64_t same = __ballot(valid);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const uint64_t ones = __ballot(valid && ((d >> b) & 1));
    same &= ((d >> b) & 1) ? ones : ~ones;
  }
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  const int rank_in_wave = __popcll(same & below);
  // the last lane of each digit group records the group's size
  if (valid && (same >> lane) == 1ull) wave_count[wv][d] = __popcll(same);
  __syncthreads();
  if (!valid) return;
  int before = rank_in_wave;
  for (int w = 0; w < wv; ++w) before += wave_count[w][d];
  const int64_t at = offsets[(int64_t)d * ntiles + blockIdx.x] + before;
  keys_out[at] = key;
  vals_out[at] = vals_in[i];
}

__global__ __launch_bounds__(256) void copy_pairs_kernel(const uint32_t* k, const int32_t* v, int64_t n,
                                                         uint32_t* k2, int32_t* v2) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  k2[i] = k[i];
  v2[i] = v[i];
}

}  // namespace

int64_t task_order_table_size(int64_t n) {
  int64_t s = 1;
  while (s < 2 * n) s <<= 1;
  return s;
}

// Work memory of the sort: the (digit, tile) histogram (int32), its offsets
// (int64, one more entry) and the scan's block sums, each 256-byte aligned.
hipError_t task_order_temp_bytes(int64_t n, size_t* bytes) {
  *bytes = 0;
  if (n <= 1) return hipSuccess;
  const int64_t m = 256 * ((n + kSortTile - 1) / kSortTile);
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  *bytes = up(sizeof(int32_t) * m) + up(sizeof(int64_t) * (m + 1)) + up(sizeof(int64_t) * scan_tmp_elems(m));
  return hipSuccess;
}

hipError_t launch_task_order(const OrderArgs& a, hipStream_t s) {
  const int64_t n = a.ntasks;
  if (n <= 1) return hipSuccess;
  // 1. representatives: the lowest task index per distinct list hash
  hipLaunchKernelGGL(table_clear_kernel, dim3(grid(a.table_size, 256)), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(task_hash_kernel, dim3(grid(n, kWavesPerBlock)), dim3(64 * kWavesPerBlock), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(representative_kernel, dim3(grid(n, 256)), dim3(256), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // 2. order by (representative, index): row order with equal lists pulled
  //    up to their first occurrence (every pass is stable, and the pairs
  //    start in index order).  The passes alternate between the two key and
  //    value buffers; the first buffer pair is chosen so that the last pass
  //    writes the order.
  const int64_t ntiles = (n + kSortTile - 1) / kSortTile, m = 256 * ntiles;
  size_t need = 0;
  if ((e = task_order_temp_bytes(n, &need)) != hipSuccess) return e;
  if (a.temp_bytes < need) return hipErrorInvalidValue;
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  uint8_t* t8 = static_cast<uint8_t*>(a.temp);
  int32_t* hist = reinterpret_cast<int32_t*>(t8);
  int64_t* offsets = reinterpret_cast<int64_t*>(t8 + up(sizeof(int32_t) * m));
  int64_t* scan_tmp = reinterpret_cast<int64_t*>(t8 + up(sizeof(int32_t) * m) + up(sizeof(int64_t) * (m + 1)));
  const int passes = sort_passes(n);
  // pass p reads buffer pair p % 2 and writes the other; after an even
  // number of passes the result is in the pair the first pass read, so that
  // case starts from a copy in (rep_sorted, order)
  uint32_t* kbuf[2] = {a.rep, a.rep_sorted};
  int32_t* vbuf[2] = {a.idx_in, a.order};
  if (passes % 2 == 0) {
    hipLaunchKernelGGL(copy_pairs_kernel, dim3(grid(n, 256)), dim3(256), 0, s, a.rep, a.idx_in, n, a.rep_sorted,
                       a.order);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    std::swap(kbuf[0], kbuf[1]);
    std::swap(vbuf[0], vbuf[1]);
  }
  int cur = 0;
  for (int p = 0; p < passes; ++p, cur ^= 1) {
    hipLaunchKernelGGL(digit_hist_kernel, dim3((unsigned)ntiles), dim3(kSortTile), 0, s, kbuf[cur], n, 8 * p, hist,
                       ntiles);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_scan_i32(hist, offsets, m, scan_tmp, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(digit_scatter_kernel, dim3((unsigned)ntiles), dim3(kSortTile), 0, s, kbuf[cur], vbuf[cur], n,
                       8 * p, offsets, ntiles, kbuf[cur ^ 1], vbuf[cur ^ 1]);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (!a.tasks_out) return hipSuccess;
  hipLaunchKernelGGL(task_gather_kernel, dim3(grid(n, 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace bsa
