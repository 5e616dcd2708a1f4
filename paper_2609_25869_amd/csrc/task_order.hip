// Dispatch order of a segment's tasks.
//
// The attention kernel gives each XCD a contiguous range of the dispatch
// order, and an XCD holds a few dozen tasks at once that all stream K/V
// tiles through its own L2.  Two tasks share L2 lines only if they read the
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
#include <hipcub/hipcub.hpp>

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

}  // namespace

int64_t task_order_table_size(int64_t n) {
  int64_t s = 1;
  while (s < 2 * n) s <<= 1;
  return s;
}

hipError_t task_order_temp_bytes(int64_t n, size_t* bytes) {
  *bytes = 0;
  if (n <= 1) return hipSuccess;
  return hipcub::DeviceRadixSort::SortPairs(nullptr, *bytes, static_cast<const uint32_t*>(nullptr),
                                            static_cast<uint32_t*>(nullptr), static_cast<const int32_t*>(nullptr),
                                            static_cast<int32_t*>(nullptr), (int)n, 0, rep_bits(n), (hipStream_t)0);
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
  //    up to their first occurrence (the radix sort is stable)
  size_t bytes = a.temp_bytes;
  e = hipcub::DeviceRadixSort::SortPairs(a.temp, bytes, a.rep, a.rep_sorted, a.idx_in, a.order, (int)n, 0, rep_bits(n),
                                         s);
  if (e != hipSuccess || !a.tasks_out) return e;
  hipLaunchKernelGGL(task_gather_kernel, dim3(grid(n, 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace bsa
